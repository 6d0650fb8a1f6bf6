// Grouped mixed-bit expert GEMM (Sec. 3.3.2: dequantization fused with the
// expert matrix products) for any number of tokens per expert, and the
// weighted combine (Fig. 1: outputs of the activated experts weighted by the
// gate).
//
// Work is cut into tiles of (expert, bit-width bucket, 256 positions, 128
// output rows), one 512-thread workgroup each.  Positions are the (token, slot) pairs sorted by (expert,
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

constexpr int BM = 256, BN = 128, KS = 64, kThreads = 512;

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


typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 b2 __attribute__((ext_vector_type(2)));

__device__ inline h2 as_h2(uint32_t v) { return __builtin_bit_cast(h2, v); }
__device__ inline uint32_t as_u(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ inline uint32_t h2_to_bf2(h2 v) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(__builtin_convertvector(v, f2), b2));
}
__device__ inline uint32_t h2_splat(float v) {
  const _Float16 h = (_Float16)v;
  return as_u(h2{h, h});
}

// Tiles in LDS are [rows][KS] bf16 (128 bytes per row) with the 16-byte
// chunks of a row stored at chunk ^ (row & 7), so that the 16 rows an MFMA
// operand reads spread over the banks.
__device__ inline int swz(int row, int chunk) { return row * KS + ((chunk ^ (row & 7)) << 3); }

// Grouped expert GEMM: one workgroup computes BM positions x BN weight rows
// of one (expert, bit-width) bucket.
//   in:  bf16 activations, position p reads in[src_row(p) * in_ld + k] with
//        src_row = perm ? perm[p] / kdiv : p
//   SWIGLU: W is [2f][K] (w13); the tile holds 64 rows of W1 and the same 64
//           rows of W3 interleaved in 16-row slices, out = h [pos][f] bf16
//   else:   W is [N][K], out = y [pos][N] fp32
// Per K step (KS columns): the activations and the plane words, scales and
// zero points of the next step are loaded into registers while the MFMAs of
// the current step run; then each thread dequantizes 16 weights of one row
// into LDS.  Dequantization works on pairs of weights (j, j + 16) of a plane
// word in packed fp16: shifting the word left by 15 - j puts bit j at bit 15
// and bit j + 16 at bit 31, the sign positions of the two halves, and v_bfi
// turns the pair into (+-c_p, +-c_p).  With every plane read as a sign,
//   W^_b = s1 (Q - z) + sum_{p>=b_min} s_p sigma_p
//        = C + sum_{p<b} c_p (2 bit_p - 1),  c_p = s1 2^(p-1) for p < b_min,
//          c_p = s_p for p >= b_min,  C = s1 ((2^b_min - 1) / 2 - z),
// accumulated in fp16 from C, then rounded to bf16 for the MFMA.
template <int G, bool SWIGLU>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const uint16_t* __restrict__ in, int in_ld,
                                                        const int32_t* __restrict__ perm, int kdiv,
                                                        MwqView W, int expert_fixed, Sched sc,
                                                        int f, int N, void* __restrict__ out,
                                                        int out_ld) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[BM * KS];
  __shared__ __attribute__((aligned(16))) uint16_t ws[BN * KS];
  __shared__ int s_info[4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // ---- which bucket / tile ----
  if (tid == 0) {
    int j = 0, nb = sc.nb;
    int mt = blockIdx.y;
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
  const int n0 = blockIdx.x * (SWIGLU ? BN / 2 : BN);  // first output row
  const int K = W.cols, BR = W.BR(), b_min = W.b_min;

  // ---- activation loader: row xr, 16-byte chunks 4 xh .. 4 xh + 3 ----
  const int xr = tid >> 1, xh = tid & 1;
  const uint16_t* xsrc = nullptr;
  if (xr < cnt) {
    const int pos = pos0 + xr;
    xsrc = in + (size_t)(perm ? perm[pos] / kdiv : pos) * in_ld + 32 * xh;
  }
  // ---- dequantizer: tile row dc, 32-column word dsub, pairs 8 dh .. 8 dh + 7 ----
  const int item = tid >> 1, dh = tid & 1;
  const int dc = item >> 1, dsub = item & 1;
  int mrow;  // matrix row of tile row dc
  bool drow_ok;
  if (SWIGLU) {
    const int dwn = dc >> 6, cc = dc & 63, sl = cc >> 4;
    const int hrow = n0 + 32 * dwn + 16 * (sl >> 1) + (cc & 15);
    drow_ok = hrow < f;
    mrow = ((sl & 1) ? f : 0) + hrow;
  } else {
    mrow = n0 + dc;
    drow_ok = mrow < N;
  }
  const int drb = drow_ok ? mrow / BR : 0, dib = drow_ok ? mrow % BR : 0;
  uint32_t sh_m;  // opaque copy of the sign mask: keeps v_bfi on registers
  asm volatile("" : "=v"(sh_m) : "0"(0x80008000u));

  uint4 xreg[4];
  uint32_t preg[8];
  uint16_t sreg[8];
  uint32_t zreg = 0;
  auto load_step = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      xreg[i] = xsrc ? *(const uint4*)(xsrc + k0 + 8 * i) : uint4{0u, 0u, 0u, 0u};
    if (drow_ok) {
      const size_t blk = W.block(expert, drb, k0 / G);
      const int wq = ((k0 % G) / 32 + dsub) * BR + dib;
#pragma unroll
      for (int p = 0; p < 8; ++p)
        if (p < bits) preg[p] = W.planes[W.plane_word(blk, p, wq)];
#pragma unroll
      for (int l = 0; l < 8; ++l)
        if (l < bits - b_min + 1) sreg[l] = W.scales[W.scale_idx(blk, l, dib)];
      zreg = W.zeros[W.zero_idx(blk, dib)];
    }
  };
  auto store_step = [&]() {
    // activations
    uint4* xd = (uint4*)xs;
#pragma unroll
    for (int i = 0; i < 4; ++i) xd[swz(xr, 4 * xh + i) >> 3] = xreg[i];
    // weights
    uint32_t lo[4], hi[4];
    if (drow_ok) {
      const float s1 = h2f(sreg[0]);
      uint32_t cp[8];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const float c = p < b_min ? s1 * (float)(1 << p) * 0.5f : (p < bits ? h2f(sreg[p - b_min + 1]) : 0.0f);
        cp[p] = h2_splat(c) & 0x7fff7fffu;
      }
      const uint32_t C = h2_splat(s1 * ((float)((1 << b_min) - 1) * 0.5f - (float)zreg));
      h2 acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = as_h2(C);
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        if (p >= bits) break;  // uniform
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint32_t t = preg[p] << (15 - (8 * dh + j));
          const uint32_t v = (sh_m & t) | (~sh_m & cp[p]);  // bit set -> -c_p
          acc[j] = acc[j] - as_h2(v);
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t a = h2_to_bf2(acc[2 * j]), b = h2_to_bf2(acc[2 * j + 1]);
        lo[j] = (a & 0xffffu) | (b << 16);          // weights 8 dh + 2j, +1
        hi[j] = (a >> 16) | (b & 0xffff0000u);      // weights 16 + 8 dh + 2j, +1
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) lo[j] = hi[j] = 0u;
    }
    uint4* wd = (uint4*)ws;
    wd[swz(dc, 4 * dsub + dh) >> 3] = uint4{lo[0], lo[1], lo[2], lo[3]};
    wd[swz(dc, 4 * dsub + 2 + dh) >> 3] = uint4{hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nsteps = K / KS;
  load_step(0);
  store_step();
  __syncthreads();
  for (int st = 0; st < nsteps; ++st) {
    if (st + 1 < nsteps) load_step((st + 1) * KS);
#pragma unroll
    for (int kk = 0; kk < KS / 32; ++kk) {
      bf16x8 bfr[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int col = 64 * wn + 16 * nt + (lane & 15);
        bfr[nt] = *(const bf16x8*)(ws + swz(col, 4 * kk + (lane >> 4)));
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = 64 * wm + 16 * mt + (lane & 15);
        const bf16x8 afr = *(const bf16x8*)(xs + swz(row, 4 * kk + (lane >> 4)));
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afr, bfr[nt], acc[mt][nt], 0, 0, 0);
      }
    }
    __syncthreads();
    if (st + 1 < nsteps) {
      store_step();
      __syncthreads();
    }
  }

  // ---- epilogue ----
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 64 * wm + 16 * mt + 4 * (lane >> 4) + r;
      if (m >= cnt) continue;
      const size_t pos = (size_t)(pos0 + m);
      if (SWIGLU) {
#pragma unroll
        for (int sp = 0; sp < 2; ++sp) {
          const int n = n0 + 32 * wn + 16 * sp + (lane & 15);
          if (n >= f) continue;
          const float a = acc[mt][2 * sp][r], c = acc[mt][2 * sp + 1][r];
          ((uint16_t*)out)[pos * out_ld + n] = f2bf(silu(a) * c);
        }
      } else {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const int n = n0 + 64 * wn + 16 * nt + (lane & 15);
          if (n >= N) continue;
          ((float*)out)[pos * out_ld + n] = acc[mt][nt][r];
        }
      }
    }
  }
}

// fp32 activations are rounded to bf16 once for the GEMM's operand tiles.
__global__ void to_bf16_kernel(const float* __restrict__ in, size_t n, uint16_t* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = f2bf(in[i]);
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

template <bool SWIGLU>
hipError_t run_gemm(const uint16_t* in, int in_ld, const int32_t* perm, int kdiv, const MwqView& W,
                    int expert_fixed, const Sched& sc, int mtiles_ub, int f, void* out, int out_ld,
                    hipStream_t s) {
  const int N = SWIGLU ? W.rows / 2 : W.rows;
  const int per = SWIGLU ? BN / 2 : BN;
  // output-row tiles vary fastest: consecutive workgroups, which the
  // dispatcher deals round-robin to the 8 XCDs, share one M-tile, so every
  // XCD's L2 holds the activations of the one or two M-tiles in flight
  // rather than of all of them
  dim3 grid((N + per - 1) / per, mtiles_ub);
  if (mtiles_ub <= 0) return hipSuccess;
  if (W.group == 128)
    gemm_kernel<128, SWIGLU><<<grid, kThreads, 0, s>>>(in, in_ld, perm, kdiv, W, expert_fixed, sc,
                                                       f, N, out, out_ld);
  else
    gemm_kernel<64, SWIGLU><<<grid, kThreads, 0, s>>>(in, in_ld, perm, kdiv, W, expert_fixed, sc,
                                                      f, N, out, out_ld);
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
  L.xb_off = off;     off += align256(sizeof(uint16_t) * (size_t)T * d);
  const size_t nd = T <= kDecodeMaxTokens ? (size_t)T * k : 0;  // decode positions
  // decode work list: at most one run per active expert plus one per 8 positions
  L.elist_off = off;  off += align256(sizeof(int32_t) * (4 * ((size_t)E + (nd + 7) / 8) + 4));
  const size_t nz = nd ? nd + 1 : 0;  // plus one all-zero activation slot
  L.xq13_off = off;   off += align256(nz * d * 2);
  const size_t nxs = nz ? nz + 8 : 0;  // info words, padded for 8-position reads
  L.xs13_off = off;   off += align256(nxs * sizeof(uint32_t));
  L.h32_off = off;    off += align256(nd * d_ff * sizeof(float));
  L.xq2_off = off;    off += align256(nz * d_ff * 2);
  L.xs2_off = off;    off += align256(nxs * sizeof(uint32_t));
  // partial maxima of |h|: one word per (position, 16-row block of d_ff)
  L.hmax_off = off;   off += align256(nd * ((size_t)(d_ff + 15) / 16) * sizeof(uint32_t));
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
  // bf16 activations for the grouped GEMM (fp32 inputs are rounded once)
  const uint16_t* xb = (const uint16_t*)x;
  const bool gemm_needed = has_shared || !decode_path_ok(w13, w2, T);
  if (xd == D2MOE_F32 && gemm_needed) {
    uint16_t* xw = (uint16_t*)(base + L.xb_off);
    const size_t n = (size_t)T * d;
    to_bf16_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>((const float*)x, n, xw);
    hipError_t e0 = hipGetLastError();
    if (e0 != hipSuccess) return e0;
    xb = xw;
  }

  hipError_t err;
  if (decode_path_ok(w13, w2, T)) {
    DecodeBuffers db;
    db.elist = (int32_t*)(base + L.elist_off);
    db.xq13 = (uint8_t*)(base + L.xq13_off);
    db.xs13 = (uint32_t*)(base + L.xs13_off);
    db.h32 = (float*)(base + L.h32_off);
    db.xq2 = (uint8_t*)(base + L.xq2_off);
    db.xs2 = (uint32_t*)(base + L.xs2_off);
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
    err = run_gemm<true>(xb, d, r->perm, k, W13, 0, sc, ub, d_ff, h, d_ff, s);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[1], s)) != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[2], s)) != hipSuccess) return err;
    err = run_gemm<false>(h, d_ff, nullptr, 1, W2, 0, sc, ub, d_ff, y, d, s);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[3], s)) != hipSuccess) return err;
  }

  if (has_shared) {
    Sched one{nullptr, nullptr, nullptr, 0, T, shared_bits, 1, sw13->b_min};
    const int ubs = (T + BM - 1) / BM;
    const MwqView S13 = view_of(sw13), S2 = view_of(sw2);
    err = run_gemm<true>(xb, d, nullptr, 1, S13, 0, one, ubs, shared_d_ff, hs, shared_d_ff, s);
    if (err != hipSuccess) return err;
    err = run_gemm<false>(hs, shared_d_ff, nullptr, 1, S2, 0, one, ubs, shared_d_ff, ys, d, s);
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
