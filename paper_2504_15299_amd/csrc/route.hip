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

// Sum over the wave, valid in lane 0: each row of 16 lanes is summed with DPP
// row shifts (lane i adds lane i + 8, + 4, + 2, + 1), then lane 0 adds the
// four row sums pairwise.  Six additions per term, as in a shuffle
// butterfly, without the LDS permute path.
__device__ inline float wave_sum_lane0(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x108, 0xf, 0xf, true));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x104, 0xf, 0xf, true));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x102, 0xf, 0xf, true));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x101, 0xf, 0xf, true));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (v + r1) + (r2 + r3);
}
__device__ inline float load1(const uint16_t* p) { return bf2f(*p); }

// logits[t][e] = x[t] . Wg[e] (+ bias[e]) for a tile of TT tokens by EE
// experts per workgroup.  Each thread takes 8 consecutive columns per step
// (one 16-byte load of x per token, two of each gate row) with one fp32 fma
// chain per (token, expert); the partial sums are reduced across the wave
// (DPP row shifts, then the four rows) and across the waves through LDS.  A
// term passes through at most ceil(d/256) + 11 roundings.  Small batches use 1 x 1 tiles, so that
// many workgroups share the loads and every one of them is short; large
// batches use 4 x 8 tiles, which read each gate row once per four tokens.
template <typename XT, int TT, int EE>
__global__ __launch_bounds__(kGateThreads) void gate_kernel(
    const XT* __restrict__ x, int T, int d, const float* __restrict__ Wg,
    const float* __restrict__ bias, int E, float* __restrict__ logits) {
  constexpr int NWAVE = kGateThreads / 64;
  __shared__ float part[NWAVE][TT * EE];
  const int t0 = blockIdx.x * TT, e0 = blockIdx.y * EE;
  const int nt = T - t0 < TT ? T - t0 : TT, ne = E - e0 < EE ? E - e0 : EE;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // rows past the tile's end repeat its last row; their sums are not written
  const XT* xr[TT];
  const float* wr[EE];
#pragma unroll
  for (int i = 0; i < TT; ++i) xr[i] = x + (size_t)(t0 + (i < nt ? i : nt - 1)) * d;
#pragma unroll
  for (int j = 0; j < EE; ++j) wr[j] = Wg + (size_t)(e0 + (j < ne ? j : ne - 1)) * d;
  const bool vec = (d & 7) == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)Wg & 15) == 0;
  float acc[TT][EE];
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int j = 0; j < EE; ++j) acc[i][j] = 0.0f;
  if (vec) {
#pragma unroll 2
    for (int c = 8 * tid; c < d; c += 8 * kGateThreads) {
      float xv[TT][8];
#pragma unroll
      for (int i = 0; i < TT; ++i) load8(xr[i] + c, xv[i]);
#pragma unroll
      for (int j = 0; j < EE; ++j) {
        float wv[8];
        load8(wr[j] + c, wv);
#pragma unroll
        for (int i = 0; i < TT; ++i)
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[i][j] = fmaf(xv[i][q], wv[q], acc[i][j]);
      }
    }
  } else {
    for (int c = tid; c < d; c += kGateThreads) {
      float xv[TT];
#pragma unroll
      for (int i = 0; i < TT; ++i) xv[i] = load1(xr[i] + c);
#pragma unroll
      for (int j = 0; j < EE; ++j) {
        const float wv = wr[j][c];
#pragma unroll
        for (int i = 0; i < TT; ++i) acc[i][j] = fmaf(xv[i], wv, acc[i][j]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int j = 0; j < EE; ++j) {
      const float v = wave_sum_lane0(acc[i][j]);
      if (lane == 0) part[wave][i * EE + j] = v;
    }
  __syncthreads();
  if (tid < TT * EE) {
    const int i = tid / EE, j = tid % EE;
    if (i < nt && j < ne) {
      float sum = 0.0f;
      for (int w = 0; w < NWAVE; ++w) sum += part[w][tid];
      logits[(size_t)(t0 + i) * E + e0 + j] = sum + (bias ? bias[e0 + j] : 0.0f);
    }
  }
}

// Top-k of one token by (logit descending, index ascending), softmax over
// the selected logits and bit-width lookup with range checks, by one wave:
// lane e holds logit e and the table's bit-width for expert e (E <= 64).
// Each of the k rounds takes the wave maximum of the remaining logits and,
// among the lanes that hold it, the lowest index; round i's choice is kept by
// lane i, which writes entry i at the end.  The softmax denominator sums the
// selected terms in selection order.  Returns the token's flag bits (1: a
// bit-width outside [b_min, b_max] was clamped, 2: a request id outside
// [0, R) was clamped), the same on every lane.
struct TopkIn {
  float v;  // this lane's logit
  int b;    // this lane's bit-width for the token
  int flag;
};

// Where each (token, expert) bit-width comes from: a per-(request, expert)
// table, or the learned bit-width routers' logits [T][E][L] over the nest's
// L = b_max - b_min + 1 widths, whose argmax (lowest width on ties) selects
// the width (Sec. 3.2).
struct BitSource {
  const int32_t* token_req;
  const uint8_t* bit_table;
  int R;
  const float* rlogits;
  int L, b_min;
};

__device__ inline TopkIn topk_load(const float* __restrict__ logits, int t, int E,
                                   const BitSource& bs, int lane) {
  TopkIn in;
  in.flag = 0;
  const bool have = lane < E;
  in.v = have ? logits[(size_t)t * E + lane] : 0.0f;
  if (bs.rlogits) {
    int best = 0;
    if (have) {
      const float* rl = bs.rlogits + ((size_t)t * E + lane) * bs.L;
      float bv = rl[0];
      for (int l = 1; l < bs.L; ++l) {
        const float v = rl[l];
        if (v > bv) {
          bv = v;
          best = l;
        }
      }
    }
    in.b = bs.b_min + best;
    return in;
  }
  int r = bs.token_req ? bs.token_req[t] : 0;
  if (r < 0 || r >= bs.R) {
    in.flag = 2;
    r = r < 0 ? 0 : bs.R - 1;
  }
  in.b = have ? (int)bs.bit_table[(size_t)r * E + lane] : 0;
  return in;
}

__device__ inline int topk_wave(const TopkIn& in, int t, int E, int k, int b_min, int b_max,
                                int lane, int32_t* __restrict__ topk_idx,
                                float* __restrict__ topk_w, uint8_t* __restrict__ topk_bits,
                                int* lkeys = nullptr, int L = 0) {
  uint64_t avail = E >= 64 ? ~0ull : ((1ull << E) - 1);
  float lmax = 0.0f, den = 0.0f;
  int my_idx = 0, my_b = 0;
  float my_v = 0.0f;
  for (int i = 0; i < k; ++i) {
    const bool live = (avail >> lane) & 1ull;
    float m = live ? in.v : -INFINITY;
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
    uint64_t cand = __ballot(live && in.v == m);
    if (cand == 0) cand = avail;  // only NaN left
    const int best = __ffsll((unsigned long long)cand) - 1;
    const float bv = __shfl(in.v, best, 64);
    const int bb = __shfl(in.b, best, 64);
    avail &= ~(1ull << best);
    if (i == 0) lmax = bv;
    den += expf(bv - lmax);
    if (lane == i) {
      my_idx = best;
      my_v = bv;
      my_b = bb;
    }
  }
  int flag = in.flag;
  const bool clamp = lane < k && (my_b < b_min || my_b > b_max);
  if (__ballot(clamp)) flag |= 1;
  if (lane < k) {
    const int b = my_b < b_min ? b_min : (my_b > b_max ? b_max : my_b);
    topk_idx[t * k + lane] = my_idx;
    topk_bits[t * k + lane] = (uint8_t)b;
    topk_w[t * k + lane] = expf(my_v - lmax) / den;
    if (lkeys) lkeys[t * k + lane] = my_idx * L + (b - b_min);  // the slot's histogram key
  }
  return flag;
}

// Batches above kInlineTopk tokens: one wave per token over many
// workgroups; each token's flag bits go to perm[t] (T <= T k entries) until
// the histogram kernel combines them and overwrites perm.
constexpr int kInlineTopk = 64;
constexpr int kTopkThreads = 256;

__global__ __launch_bounds__(kTopkThreads) void topk_kernel(
    const float* __restrict__ logits, int T, int E, int k, BitSource bs, int b_min, int b_max,
    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w, uint8_t* __restrict__ topk_bits,
    int32_t* __restrict__ tflags) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * (kTopkThreads / 64) + (threadIdx.x >> 6);
  if (t >= T) return;
  const TopkIn in = topk_load(logits, t, E, bs, lane);
  const int fl = topk_wave(in, t, E, k, b_min, b_max, lane, topk_idx, topk_w, topk_bits);
  if (lane == 0) tflags[t] = fl;
}

constexpr int kHistThreads = 1024;
constexpr int kHistWaves = kHistThreads / 64;
constexpr int kMaxKeys = 64 * 8;  // E <= 64, L <= 8

// Single workgroup: every token's top-k, softmax weights and bit-widths
// (one token per thread), then the histogram of keys (expert * L + bit -
// b_min), exclusive scan, stable placement of slots in ascending slot order
// within each key, inverse permutation and largest requested bit per expert.
// Slots are taken 1024 at a time; within a chunk the rank of a slot among
// earlier slots with the same key comes from wave ballots (equal-key lane
// masks) plus per-wave counts of earlier waves.
__global__ __launch_bounds__(kHistThreads) void hist_perm_kernel(
    const float* __restrict__ logits, int k, BitSource bs, int b_max, int32_t* __restrict__ topk_idx,
    float* __restrict__ topk_w, uint8_t* __restrict__ topk_bits, int T, int n, int E, int L,
    int b_min, int32_t* __restrict__ flags, int32_t* __restrict__ hist,
    int32_t* __restrict__ offsets, int32_t* __restrict__ perm, int32_t* __restrict__ slot_of,
    uint8_t* __restrict__ maxbit) {
  __shared__ int cnt[kMaxKeys];
  __shared__ int off[kMaxKeys + 1];
  __shared__ int run[kMaxKeys];
  __shared__ int wave_cnt[kHistWaves][kMaxKeys];
  // slot keys of the batches whose top-k runs here (T k <= 64 * 64), so that
  // the histogram and placement read them from LDS rather than back from
  // global memory
  __shared__ int lkey[kInlineTopk * 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nkeys = E * L;
  __shared__ int flag_acc;
  if (tid == 0) flag_acc = 0;
  for (int j = tid; j < nkeys; j += kHistThreads) { cnt[j] = 0; run[j] = 0; }
  __syncthreads();
  int fl = 0;
  if (T <= kInlineTopk) {
    // wave w selects for tokens w, w + 16, w + 32, w + 48, all loaded first
    constexpr int TPW = kInlineTopk / kHistWaves;
    TopkIn in[TPW];
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int t = wave + kHistWaves * j;
      if (t < T) in[j] = topk_load(logits, t, E, bs, lane);
    }
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      const int t = wave + kHistWaves * j;
      if (t < T)
        fl |= topk_wave(in[j], t, E, k, b_min, b_max, lane, topk_idx, topk_w, topk_bits, lkey, L);
    }
    if (lane != 0) fl = 0;
  } else {
    // topk_kernel left each token's flag bits in perm[t]; combine them
    // before perm is overwritten below
    for (int t = tid; t < T; t += kHistThreads) fl |= perm[t];
  }
  if (fl) atomicOr(&flag_acc, fl);
  // the barrier also orders this workgroup's global writes of the
  // selections before the reads below
  __syncthreads();
  if (tid == 0) *flags = flag_acc;
  const bool inline_keys = T <= kInlineTopk;
  for (int s = tid; s < n; s += kHistThreads)
    atomicAdd(&cnt[inline_keys ? lkey[s] : topk_idx[s] * L + (topk_bits[s] - b_min)], 1);
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
    const int key =
        !valid ? 0 : inline_keys ? lkey[s] : topk_idx[s] * L + (topk_bits[s] - b_min);
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

template <typename XT>
hipError_t run_gate(const XT* x, int T, int d, const float* Wg, const float* bias, int E,
                    float* logits, hipStream_t s) {
  if ((size_t)T * E <= 4096)
    gate_kernel<XT, 1, 1><<<dim3(T, E), kGateThreads, 0, s>>>(x, T, d, Wg, bias, E, logits);
  else
    gate_kernel<XT, 4, 8><<<dim3((T + 3) / 4, (E + 7) / 8), kGateThreads, 0, s>>>(x, T, d, Wg,
                                                                                 bias, E, logits);
  return hipGetLastError();
}

}  // namespace

static hipError_t route_common(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                               const float* bias, int E, int k, const BitSource& bs, int b_min,
                               int b_max, const d2moe_routing* out, hipStream_t s) {
  hipError_t err;
  const int L = b_max - b_min + 1;
  if (T > 0) {
    if (xd == D2MOE_BF16)
      err = run_gate((const uint16_t*)x, T, d, Wg, bias, E, out->logits, s);
    else
      err = run_gate((const float*)x, T, d, Wg, bias, E, out->logits, s);
    if (err != hipSuccess) return err;
    if (T > kInlineTopk) {
      const int per = kTopkThreads / 64;
      topk_kernel<<<(T + per - 1) / per, kTopkThreads, 0, s>>>(
          out->logits, T, E, k, bs, b_min, b_max, out->topk_idx, out->topk_w, out->topk_bits,
          out->perm);
      if ((err = hipGetLastError()) != hipSuccess) return err;
    }
  }
  hist_perm_kernel<<<1, kHistThreads, 0, s>>>(
      out->logits, k, bs, b_max, out->topk_idx, out->topk_w, out->topk_bits, T, T * k, E, L,
      b_min, out->flags, out->hist, out->offsets, out->perm, out->slot_of, out->expert_maxbit);
  return hipGetLastError();
}

hipError_t launch_route(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                        const float* bias, int E, int k, const int32_t* token_req,
                        const uint8_t* bit_table, int R, int b_min, int b_max,
                        const d2moe_routing* out, hipStream_t s) {
  const BitSource bs{token_req, bit_table, R, nullptr, b_max - b_min + 1, b_min};
  return route_common(x, xd, T, d, Wg, bias, E, k, bs, b_min, b_max, out, s);
}

hipError_t launch_route_learned(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                                const float* bias, int E, int k, const float* Wr,
                                const float* br, int b_min, int b_max, float* bit_logits,
                                const d2moe_routing* out, hipStream_t s) {
  const int L = b_max - b_min + 1;
  if (T > 0) {
    // the bit-width routers' logits, the E * L router rows taken as gate rows
    const hipError_t err =
        xd == D2MOE_BF16 ? run_gate((const uint16_t*)x, T, d, Wr, br, E * L, bit_logits, s)
                         : run_gate((const float*)x, T, d, Wr, br, E * L, bit_logits, s);
    if (err != hipSuccess) return err;
  }
  const BitSource bs{nullptr, nullptr, 1, bit_logits, L, b_min};
  return route_common(x, xd, T, d, Wg, bias, E, k, bs, b_min, b_max, out, s);
}

}  // namespace d2moe
