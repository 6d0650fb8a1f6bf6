// Dual routing (Fig. 1): gate logits, top-k expert IDs with a softmax over the
// selected logits, the bit-width of every activated expert from the
// per-(request, expert) table, and the (expert, bit-width) selection counts
// B_{j,k} of Sec. 3.4.3 with their exclusive scan and the stable permutation
// of (token, slot) pairs that the grouped expert kernels consume.
//
// Everything stays on the device; nothing synchronizes with the host.
#include "internal.h"

namespace d2moe {
namespace {

constexpr int kGateThreads = 256;
constexpr int kGateE = 8;  // experts per pass over the token's row
constexpr int kMaxExperts = 64;

__device__ inline void load8(const float* p, float (&v)[8]) {
  const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ inline void load8(const uint16_t* p, float (&v)[8]) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf2f((uint16_t)(w[i] & 0xffff));
    v[2 * i + 1] = bf2f((uint16_t)(w[i] >> 16));
  }
}
__device__ inline float load1(const float* p) { return *p; }
__device__ inline float load1(const uint16_t* p) { return bf2f(*p); }

// Top-k of one token by (logit descending, index ascending), softmax over
// the selected logits, bit-width lookup with range checks.  The token's flag
// bits (1: a bit-width outside [b_min, b_max] was clamped, 2: a request id
// outside [0, R) was clamped) go to tflags[t]; the histogram kernel combines
// them into the routing flag word.
__device__ inline void select_topk(const float* l, int t, int E, int k,
                                   const int32_t* __restrict__ token_req,
                                   const uint8_t* __restrict__ bit_table, int R, int b_min,
                                   int b_max, int32_t* __restrict__ topk_idx,
                                   float* __restrict__ topk_w, uint8_t* __restrict__ topk_bits,
                                   int32_t* __restrict__ tflags) {
  uint64_t taken = 0;
  int r = token_req ? token_req[t] : 0;
  int flag = 0;
  if (r < 0 || r >= R) {
    flag |= 2;
    r = r < 0 ? 0 : R - 1;
  }
  // selection in descending order: the first pick holds the largest logit
  float lmax = 0.0f, den = 0.0f;
  for (int i = 0; i < k; ++i) {
    int best = -1;
    for (int e = 0; e < E; ++e) {
      if ((taken >> e) & 1ull) continue;
      if (best < 0 || l[e] > l[best]) best = e;
    }
    taken |= 1ull << best;
    if (i == 0) lmax = l[best];
    den += expf(l[best] - lmax);
    topk_idx[t * k + i] = best;
    int b = bit_table[(size_t)r * E + best];
    if (b < b_min || b > b_max) {
      flag |= 1;
      b = b < b_min ? b_min : b_max;
    }
    topk_bits[t * k + i] = (uint8_t)b;
  }
  for (int i = 0; i < k; ++i) topk_w[t * k + i] = expf(l[topk_idx[t * k + i]] - lmax) / den;
  tflags[t] = flag;
}

// logits[t][e] = x[t] . Wg[e] (+ bias[e]); one workgroup per token, which
// then also takes the token's top-k (select_topk below).  Each
// thread takes 8 consecutive columns per step (one 16-byte load of x, two of
// each gate row) for up to kGateE experts per pass, with one fp32 fma chain
// per expert; the partial sums are reduced across the wave with shuffles and
// across the waves through LDS.  A term passes through at most
// ceil(d/256) + 11 roundings.
template <typename XT>
__global__ __launch_bounds__(kGateThreads) void gate_kernel(
    const XT* __restrict__ x, int d, const float* __restrict__ Wg, const float* __restrict__ bias,
    int E, int k, const int32_t* __restrict__ token_req, const uint8_t* __restrict__ bit_table,
    int R, int b_min, int b_max, float* __restrict__ logits, int32_t* __restrict__ topk_idx,
    float* __restrict__ topk_w, uint8_t* __restrict__ topk_bits, int32_t* __restrict__ tflags) {
  constexpr int NWAVE = kGateThreads / 64;
  __shared__ float part[NWAVE][kGateE];
  __shared__ float lg[kMaxExperts];
  const int t = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const XT* xt = x + (size_t)t * d;
  const bool vec = (d & 7) == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)Wg & 15) == 0;
  for (int e0 = 0; e0 < E; e0 += kGateE) {
    const int ne = E - e0 < kGateE ? E - e0 : kGateE;
    const float* w0 = Wg + (size_t)e0 * d;
    float acc[kGateE];
#pragma unroll
    for (int j = 0; j < kGateE; ++j) acc[j] = 0.0f;
    if (vec) {
      for (int c = 8 * tid; c < d; c += 8 * kGateThreads) {
        float xv[8];
        load8(xt + c, xv);
#pragma unroll
        for (int j = 0; j < kGateE; ++j) {
          if (j >= ne) continue;  // uniform
          float wv[8];
          load8(w0 + (size_t)j * d + c, wv);
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[j] = fmaf(xv[i], wv[i], acc[j]);
        }
      }
    } else {
      for (int c = tid; c < d; c += kGateThreads) {
        const float xv = load1(xt + c);
#pragma unroll
        for (int j = 0; j < kGateE; ++j)
          if (j < ne) acc[j] = fmaf(xv, w0[(size_t)j * d + c], acc[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < kGateE; ++j)
      for (int off = 32; off > 0; off >>= 1) acc[j] += __shfl_xor(acc[j], off, 64);
    if (lane == 0) {
#pragma unroll
      for (int j = 0; j < kGateE; ++j) part[wave][j] = acc[j];
    }
    __syncthreads();
    if (tid < ne) {
      float sum = 0.0f;
      for (int w = 0; w < NWAVE; ++w) sum += part[w][tid];
      const float v = sum + (bias ? bias[e0 + tid] : 0.0f);
      logits[(size_t)t * E + e0 + tid] = v;
      lg[e0 + tid] = v;
    }
    __syncthreads();
  }
  if (tid == 0)
    select_topk(lg, t, E, k, token_req, bit_table, R, b_min, b_max, topk_idx, topk_w, topk_bits,
                tflags);
}


constexpr int kHistThreads = 1024;
constexpr int kHistWaves = kHistThreads / 64;
constexpr int kMaxKeys = 64 * 8;  // E <= 64, L <= 8

// Single workgroup: histogram of keys (expert * L + bit - b_min), exclusive
// scan, stable placement of slots in ascending slot order within each key,
// inverse permutation and largest requested bit per expert.  Slots are taken
// 1024 at a time; within a chunk the rank of a slot among earlier slots with
// the same key comes from wave ballots (equal-key lane masks) plus per-wave
// counts of earlier waves.
__global__ __launch_bounds__(kHistThreads) void hist_perm_kernel(
    const int32_t* __restrict__ topk_idx, const uint8_t* __restrict__ topk_bits, int T, int n,
    int E, int L, int b_min, int32_t* __restrict__ flags, int32_t* __restrict__ hist,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ slot_of,
    uint8_t* __restrict__ maxbit) {
  __shared__ int cnt[kMaxKeys];
  __shared__ int off[kMaxKeys + 1];
  __shared__ int run[kMaxKeys];
  __shared__ int wave_cnt[kHistWaves][kMaxKeys];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nkeys = E * L;
  __shared__ int flag_acc;
  if (tid == 0) flag_acc = 0;
  for (int j = tid; j < nkeys; j += kHistThreads) { cnt[j] = 0; run[j] = 0; }
  __syncthreads();
  // the gate kernel left each token's flag bits in perm[t]; combine them
  // before perm is overwritten below
  int fl = 0;
  for (int t = tid; t < T; t += kHistThreads) fl |= perm[t];
  if (fl) atomicOr(&flag_acc, fl);
  __syncthreads();
  if (tid == 0) *flags = flag_acc;
  for (int s = tid; s < n; s += kHistThreads)
    atomicAdd(&cnt[topk_idx[s] * L + (topk_bits[s] - b_min)], 1);
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int j = 0; j < nkeys; ++j) { off[j] = acc; acc += cnt[j]; }
    off[nkeys] = acc;
  }
  __syncthreads();
  for (int j = tid; j < nkeys; j += kHistThreads) hist[j] = cnt[j];
  for (int j = tid; j <= nkeys; j += kHistThreads) offsets[j] = off[j];
  for (int e = tid; e < E; e += kHistThreads) {
    int mb = 0;
    for (int j = 0; j < L; ++j) if (cnt[e * L + j] > 0) mb = b_min + j;
    maxbit[e] = (uint8_t)mb;
  }

  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int base = 0; base < n; base += kHistThreads) {
    for (int j = tid; j < kHistWaves * nkeys; j += kHistThreads)
      wave_cnt[j / nkeys][j % nkeys] = 0;
    __syncthreads();
    const int s = base + tid;
    const bool valid = s < n;
    const int key = valid ? topk_idx[s] * L + (topk_bits[s] - b_min) : 0;
    uint64_t same = __ballot(valid);
    for (int bit = 0; bit < 10; ++bit) {
      const bool b = (key >> bit) & 1;
      const uint64_t mb = __ballot(b);
      same &= b ? mb : ~mb;
    }
    const int rank_in_wave = __popcll(same & lt_mask);
    if (valid && rank_in_wave == 0) wave_cnt[wave][key] = __popcll(same);
    __syncthreads();
    if (valid) {
      int pos = off[key] + run[key] + rank_in_wave;
      for (int w = 0; w < wave; ++w) pos += wave_cnt[w][key];
      perm[pos] = s;
      slot_of[s] = pos;
    }
    __syncthreads();
    for (int j = tid; j < nkeys; j += kHistThreads) {
      int acc = 0;
      for (int w = 0; w < kHistWaves; ++w) acc += wave_cnt[w][j];
      run[j] += acc;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_route(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                        const float* bias, int E, int k, const int32_t* token_req,
                        const uint8_t* bit_table, int R, int b_min, int b_max,
                        const d2moe_routing* out, hipStream_t s) {
  hipError_t err;
  const int L = b_max - b_min + 1;
  if (T > 0) {
    // each token's flag bits travel in perm[t] (T <= T*k entries) until the
    // histogram kernel overwrites perm
    if (xd == D2MOE_BF16)
      gate_kernel<uint16_t><<<T, kGateThreads, 0, s>>>(
          (const uint16_t*)x, d, Wg, bias, E, k, token_req, bit_table, R, b_min, b_max,
          out->logits, out->topk_idx, out->topk_w, out->topk_bits, out->perm);
    else
      gate_kernel<float><<<T, kGateThreads, 0, s>>>(
          (const float*)x, d, Wg, bias, E, k, token_req, bit_table, R, b_min, b_max, out->logits,
          out->topk_idx, out->topk_w, out->topk_bits, out->perm);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  hist_perm_kernel<<<1, kHistThreads, 0, s>>>(out->topk_idx, out->topk_bits, T, T * k, E, L, b_min,
                                              out->flags, out->hist, out->offsets, out->perm, out->slot_of,
                                              out->expert_maxbit);
  return hipGetLastError();
}

}  // namespace d2moe
