// Grouped mixed-bit expert GEMM (Sec. 3.3.2: dequantization fused with the
// expert matrix products) for any number of tokens per expert, and the
// weighted combine (Fig. 1: outputs of the activated experts weighted by the
// gate).
//
// Work is cut into tiles of (expert, bit-width bucket, 64 positions, 64
// output rows).  Positions are the (token, slot) pairs sorted by (expert,
// bit-width), so every tile reads its expert's planes 0..b-1 only.  Per K step
// (one quantization group) the workgroup stages the gathered activations and
// the dequantized weight tile as bf16 in LDS and runs v_mfma_f32_16x16x32_bf16
// with fp32 accumulation.  The W1/W3 variant interleaves 16-row slices of W1
// and W3 so each lane holds a and c of the same output and applies SwiGLU in
// registers.
#include "internal.h"

namespace d2moe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 64, BN = 64, kThreads = 256;

// Bucket table produced on the device from the routing histogram.
struct Sched {
  const int32_t* tstart;  // [nb+1] first M-tile of each bucket (prefix sums)
  const int32_t* bstart;  // [nb] first position of each bucket
  const int32_t* bcnt;    // [nb] positions in the bucket
  int nb;                 // buckets; 0 = one bucket given by the scalars below
  int one_cnt, one_bit;   // single-bucket mode (shared expert: all tokens)
  int L, b_min;
};

__global__ void schedule_kernel(const int32_t* __restrict__ hist,
                                const int32_t* __restrict__ offsets, int nb,
                                int32_t* __restrict__ tstart, int32_t* __restrict__ bstart,
                                int32_t* __restrict__ bcnt) {
  if (threadIdx.x != 0) return;
  int acc = 0;
  for (int j = 0; j < nb; ++j) {
    tstart[j] = acc;
    bstart[j] = offsets[j];
    bcnt[j] = hist[j];
    acc += (hist[j] + BM - 1) / BM;
  }
  tstart[nb] = acc;
}

__device__ inline float silu(float a) { return a / (1.0f + __expf(-a)); }

template <typename T>
__device__ inline float ld_in(const T* p);
template <>
__device__ inline float ld_in<float>(const float* p) { return *p; }
template <>
__device__ inline float ld_in<uint16_t>(const uint16_t* p) { return bf2f(*p); }

// in:  activations, row r of the tile reads in[src_row(pos) * in_ld + k]
//      with src_row = perm ? perm[pos] / kdiv : pos
// SWIGLU: W is [2f][K] (w13), output h[pos][n] bf16, n in [0, f)
// else:   W is [N][K], output y[pos][n] f32
template <int G, bool SWIGLU, typename TIN>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const TIN* __restrict__ in, int in_ld,
                                                        const int32_t* __restrict__ perm, int kdiv,
                                                        MwqView W, int expert_fixed, Sched sc,
                                                        int f, void* __restrict__ out,
                                                        int out_ld) {
  constexpr int LDK = G + 8;  // padded LDS row (bf16 elements)
  __shared__ __attribute__((aligned(16))) uint16_t xs[BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t ws[BN * LDK];
  __shared__ int s_info[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- which bucket / tile ----
  if (tid == 0) {
    int j = 0, nb = sc.nb;
    int mt = blockIdx.x;
    if (nb == 0) {
      const int ntiles = (sc.one_cnt + BM - 1) / BM;
      s_info[0] = mt < ntiles ? 1 : 0;
      s_info[1] = mt * BM;
      s_info[2] = min(BM, sc.one_cnt - mt * BM);
      s_info[3] = sc.one_bit;
    } else if (mt >= sc.tstart[nb]) {
      s_info[0] = 0;
    } else {
      int lo = 0, hi = nb - 1;  // largest j with tstart[j] <= mt
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (sc.tstart[mid] <= mt) lo = mid; else hi = mid - 1;
      }
      j = lo;
      const int local = mt - sc.tstart[j];
      s_info[0] = 1;
      s_info[1] = sc.bstart[j] + local * BM;
      s_info[2] = min(BM, sc.bcnt[j] - local * BM);
      s_info[3] = sc.b_min + (j % sc.L);
      s_info[0] |= (j / sc.L) << 1;  // expert in the upper bits
    }
  }
  __syncthreads();
  if (!(s_info[0] & 1)) return;
  const int expert = sc.nb == 0 ? expert_fixed : (s_info[0] >> 1);
  const int pos0 = s_info[1], cnt = s_info[2], bits = s_info[3];
  const int n0 = blockIdx.y * (SWIGLU ? BN / 2 : BN);  // first output row
  const int K = W.cols, BR = W.BR();

  f32x4 acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // source row of each staged activation row (fixed over K)
  const int xm = tid >> 2, xpart = tid & 3;  // 64 rows x 4 parts
  long src_row = -1;
  if (xm < cnt) {
    const int pos = pos0 + xm;
    src_row = perm ? (long)(perm[pos] / kdiv) : (long)pos;
  }

  // tile column c (0..63) -> matrix row of W
  auto tile_row = [&](int c) -> int {
    if (SWIGLU) {
      const int w_n = c >> 5, h = (c >> 4) & 1, r = c & 15;
      return (h ? f : 0) + n0 + 16 * w_n + r;
    }
    return n0 + c;
  };

  for (int kb = 0; kb < K / G; ++kb) {
    // ---- stage activations (bf16) ----
    {
      constexpr int PER = G / 4;
      uint16_t* dst = xs + xm * LDK + xpart * PER;
      if (src_row >= 0) {
        const TIN* s = in + (size_t)src_row * in_ld + (size_t)kb * G + xpart * PER;
#pragma unroll
        for (int j = 0; j < PER; ++j) dst[j] = f2bf(ld_in<TIN>(s + j));
      } else {
#pragma unroll
        for (int j = 0; j < PER; ++j) dst[j] = 0;
      }
    }
    // ---- dequantize the weight tile (bf16) ----
    {
      const int words = BN * G / 32;  // words per plane in the tile
      for (int wi = tid; wi < words; wi += kThreads) {
        // wi enumerates (tile row block, word) ; each word = one row, 32 cols
        const int rbl = wi / 64, w = wi % 64;
        const int i = w % BR, sub = w / BR;
        const int c_first = rbl * BR;           // tile column of row-block start
        const int c = c_first + i;              // tile column of this row
        const int n = tile_row(c);
        const size_t blk = W.block(expert, n / BR, kb);
        const int ib = n % BR;                  // row within the matrix block
        const int wq = sub * BR + ib;
        const float s1 = h2f(W.scales[W.scale_idx(blk, 0, ib)]);
        const float z = (float)W.zeros[W.zero_idx(blk, ib)];
        uint32_t pw[8];
#pragma unroll
        for (int p = 0; p < 8; ++p) pw[p] = p < bits ? W.planes[W.plane_word(blk, p, wq)] : 0u;
        float sl[8];
#pragma unroll
        for (int p = 0; p < 8; ++p)
          sl[p] = (p >= W.b_min && p < bits) ? h2f(W.scales[W.scale_idx(blk, p - W.b_min + 1, ib)])
                                             : 0.0f;
        uint32_t packed[16];
#pragma unroll
        for (int j = 0; j < 32; j += 2) {
          float v2[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int jj = j + u;
            int q = 0;
#pragma unroll
            for (int p = 0; p < 8; ++p)
              if (p < W.b_min) q |= (int)((pw[p] >> jj) & 1u) << p;
            float v = ((float)q - z) * s1;
#pragma unroll
            for (int p = 0; p < 8; ++p)
              if (p >= W.b_min && p < bits) v += ((pw[p] >> jj) & 1u) ? sl[p] : -sl[p];
            v2[u] = v;
          }
          packed[j / 2] = (uint32_t)f2bf(v2[0]) | ((uint32_t)f2bf(v2[1]) << 16);
        }
        uint4* dst = (uint4*)(ws + c * LDK + sub * 32);
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          dst[q4] = uint4{packed[4 * q4], packed[4 * q4 + 1], packed[4 * q4 + 2], packed[4 * q4 + 3]};
      }
    }
    __syncthreads();
    // ---- MFMA over the group ----
#pragma unroll
    for (int kk = 0; kk < G / 32; ++kk) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        const int row = wm * 32 + t2 * 16 + (lane & 15);
        a[t2] = *(const bf16x8*)(xs + row * LDK + kk * 32 + 8 * (lane >> 4));
        const int col = wn * 32 + t2 * 16 + (lane & 15);
        b[t2] = *(const bf16x8*)(ws + col * LDK + kk * 32 + 8 * (lane >> 4));
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
    }
    __syncthreads();
  }

  // ---- epilogue ----
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = wm * 32 + mt * 16 + 4 * (lane >> 4) + r;
      if (m >= cnt) continue;
      const size_t pos = (size_t)(pos0 + m);
      if (SWIGLU) {
        const float a = acc[mt][0][r], c = acc[mt][1][r];
        const int n = n0 + 16 * wn + (lane & 15);
        ((uint16_t*)out)[pos * out_ld + n] = f2bf(silu(a) * c);
      } else {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int n = n0 + wn * 32 + nt * 16 + (lane & 15);
          ((float*)out)[pos * out_ld + n] = acc[mt][nt][r];
        }
      }
    }
  }
}

// out[t][c] = sum_i w[t][i] * y[slot_of[t*k+i]][c] (+ ys[t][c]), i ascending.
template <typename TOUT>
__global__ void combine_kernel(const float* __restrict__ y, const float* __restrict__ ys,
                               const float* __restrict__ topk_w,
                               const int32_t* __restrict__ slot_of, int k, int d,
                               TOUT* __restrict__ out) {
  const int t = blockIdx.y;
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= d) return;
  float acc = 0.0f;
  for (int i = 0; i < k; ++i) {
    const int pos = slot_of[t * k + i];
    acc += topk_w[t * k + i] * y[(size_t)pos * d + c];
  }
  if (ys) acc += ys[(size_t)t * d + c];
  if constexpr (sizeof(TOUT) == 2)
    out[(size_t)t * d + c] = f2bf(acc);
  else
    out[(size_t)t * d + c] = acc;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

template <bool SWIGLU, typename TIN>
hipError_t run_gemm(const TIN* in, int in_ld, const int32_t* perm, int kdiv, const MwqView& W,
                    int expert_fixed, const Sched& sc, int mtiles_ub, int f, void* out, int out_ld,
                    hipStream_t s) {
  const int N = SWIGLU ? W.rows / 2 : W.rows;
  dim3 grid(mtiles_ub, SWIGLU ? N / (BN / 2) : N / BN);
  if (mtiles_ub <= 0) return hipSuccess;
  if (W.group == 128)
    gemm_kernel<128, SWIGLU, TIN><<<grid, kThreads, 0, s>>>(in, in_ld, perm, kdiv, W, expert_fixed,
                                                            sc, f, out, out_ld);
  else
    gemm_kernel<64, SWIGLU, TIN><<<grid, kThreads, 0, s>>>(in, in_ld, perm, kdiv, W, expert_fixed,
                                                           sc, f, out, out_ld);
  return hipGetLastError();
}

}  // namespace

FwdWorkspace fwd_workspace_layout(int T, int d, int d_ff, int E, int k, int shared_d_ff) {
  FwdWorkspace L;
  const size_t nb = (size_t)E * 8 + 1;
  size_t off = 0;
  L.sched_off = off;  off += align256(sizeof(int32_t) * (4 * nb + 4));
  L.h_off = off;      off += align256(sizeof(uint16_t) * (size_t)T * k * d_ff);
  L.hs_off = off;     off += align256(sizeof(uint16_t) * (size_t)T * shared_d_ff);
  L.y_off = off;      off += align256(sizeof(float) * (size_t)T * k * d);
  L.ys_off = off;     off += align256(sizeof(float) * (size_t)T * (shared_d_ff > 0 ? d : 0));
  const size_t nd = T <= kDecodeMaxTokens ? (size_t)T * k : 0;  // decode positions
  // decode work list: at most one run per active expert plus one per 8 positions
  L.elist_off = off;  off += align256(sizeof(int32_t) * (4 * ((size_t)E + (nd + 7) / 8) + 4));
  const size_t nz = nd ? nd + 1 : 0;  // plus one all-zero activation slot
  L.xq13_off = off;   off += align256(nz * d * 2);
  L.xs13_off = off;   off += align256(nz * 2);
  L.h32_off = off;    off += align256(nd * d_ff * sizeof(float));
  L.xq2_off = off;    off += align256(nz * d_ff * 2);
  L.xs2_off = off;    off += align256(nz * 2);
  L.hmax_off = off;   off += align256(nz * sizeof(uint32_t));
  L.total = off;
  return L;
}

hipError_t launch_forward(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                          const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                          const d2moe_mwq* sw13, const d2moe_mwq* sw2, int shared_bits,
                          int shared_d_ff, void* out, void* ws, hipStream_t s,
                          const hipEvent_t* events) {
  if (T == 0) return hipSuccess;
  const bool has_shared = sw13 != nullptr;
  const FwdWorkspace L = fwd_workspace_layout(T, d, d_ff, E, k, has_shared ? shared_d_ff : 0);
  char* base = (char*)ws;
  const int Lv = w13->b_max - w13->b_min + 1;
  const int nb = E * Lv;
  int32_t* tstart = (int32_t*)(base + L.sched_off);
  int32_t* bstart = tstart + (nb + 1);
  int32_t* bcnt = bstart + nb;
  uint16_t* h = (uint16_t*)(base + L.h_off);
  uint16_t* hs = (uint16_t*)(base + L.hs_off);
  float* y = (float*)(base + L.y_off);
  float* ys = (float*)(base + L.ys_off);

  hipError_t err;
  if (decode_path_ok(w13, w2, T)) {
    DecodeBuffers db;
    db.elist = (int32_t*)(base + L.elist_off);
    db.ecount = db.elist + 4 * ((size_t)E + ((size_t)T * k + 7) / 8);
    db.xq13 = (uint8_t*)(base + L.xq13_off);
    db.xs13 = (uint8_t*)(base + L.xs13_off);
    db.h32 = (float*)(base + L.h32_off);
    db.xq2 = (uint8_t*)(base + L.xq2_off);
    db.xs2 = (uint8_t*)(base + L.xs2_off);
    db.hmax = (uint32_t*)(base + L.hmax_off);
    db.y = y;
    err = launch_decode_ffn(x, xd, T, d, d_ff, E, k, w13, w2, r, db, s, events);
    if (err != hipSuccess) return err;
  } else {
    schedule_kernel<<<1, 64, 0, s>>>(r->hist, r->offsets, nb, tstart, bstart, bcnt);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    Sched sc{tstart, bstart, bcnt, nb, 0, 0, Lv, w13->b_min};
    const int n = T * k;
    const int ub = (n + BM - 1) / BM + (nb < n ? nb : n);
    const MwqView W13 = view_of(w13), W2 = view_of(w2);
    if (events && (err = hipEventRecord(events[0], s)) != hipSuccess) return err;
    if (xd == D2MOE_BF16)
      err = run_gemm<true, uint16_t>((const uint16_t*)x, d, r->perm, k, W13, 0, sc, ub, d_ff, h,
                                     d_ff, s);
    else
      err = run_gemm<true, float>((const float*)x, d, r->perm, k, W13, 0, sc, ub, d_ff, h, d_ff,
                                  s);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[1], s)) != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[2], s)) != hipSuccess) return err;
    err = run_gemm<false, uint16_t>(h, d_ff, nullptr, 1, W2, 0, sc, ub, d_ff, y, d, s);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[3], s)) != hipSuccess) return err;
  }

  if (has_shared) {
    Sched one{nullptr, nullptr, nullptr, 0, T, shared_bits, 1, sw13->b_min};
    const int ubs = (T + BM - 1) / BM;
    const MwqView S13 = view_of(sw13), S2 = view_of(sw2);
    if (xd == D2MOE_BF16)
      err = run_gemm<true, uint16_t>((const uint16_t*)x, d, nullptr, 1, S13, 0, one, ubs,
                                     shared_d_ff, hs, shared_d_ff, s);
    else
      err = run_gemm<true, float>((const float*)x, d, nullptr, 1, S13, 0, one, ubs, shared_d_ff,
                                  hs, shared_d_ff, s);
    if (err != hipSuccess) return err;
    err = run_gemm<false, uint16_t>(hs, shared_d_ff, nullptr, 1, S2, 0, one, ubs, shared_d_ff, ys,
                                    d, s);
    if (err != hipSuccess) return err;
  }

  dim3 cg((d + 255) / 256, T);
  if (xd == D2MOE_BF16)
    combine_kernel<uint16_t><<<cg, 256, 0, s>>>(y, has_shared ? ys : nullptr, r->topk_w,
                                                r->slot_of, k, d, (uint16_t*)out);
  else
    combine_kernel<float><<<cg, 256, 0, s>>>(y, has_shared ? ys : nullptr, r->topk_w, r->slot_of,
                                             k, d, (float*)out);
  return hipGetLastError();
}

}  // namespace d2moe
