// Decode-regime grouped mixed-bit expert GEMV that multiplies MWQ bit-planes
// directly on the CDNA4 block-scaled matrix cores (Sec. 3.3.2: dequantization
// fused with the expert products; Sec. 3.4: low bit-widths are prefixes of
// high ones, so each expert's planes are streamed once, up to the largest
// bit-width any of its tokens requested, and every token uses the prefix it
// asked for).
//
// Per (16 rows x 128 columns) block and plane, one
// v_mfma_scale_f32_16x16x128_f8f6f4 takes
//   A: the plane as fp4 (e2m1) values +-0.5 (bit 0 -> +0.5, bit 1 -> -0.5),
//      expanded from the 32-bit plane word with two VALU ops per 8 weights;
//   B: the activations of up to 8 tokens, each as an exact pair of fp8 (e4m3)
//      pieces hi + lo with one E8M0 scale per 32 columns (16 MFMA columns).
// With A = -sigma/2 the residual bit-width b contributes s_b * sum sigma x =
// -s_b * D (A scale 2).  The base code Q = bit0 + 2 bit1 and its zero point
// fold into three chained MFMAs (planes 0 and 1 with A scales 1 and 2, plus a
// constant fp4 operand z - 1.5), so (Q - z) . x = -D as well.  Every plane
// thus costs one MFMA and one fp16-scaled FMA per output, and no weight is
// ever materialised as a number.  Tokens whose bit-width is below a plane
// skip its FMA (exec mask); they share the loads.
//
// Work split: a workgroup owns one 16-row block (W1 and the matching W3 block
// for the SwiGLU variant) of one active expert; its waves split the groups of
// the reduction dimension and reduce through LDS.  Requirements: group 128,
// b_min 2, at most 16 tokens per expert.
#include "internal.h"

namespace d2moe {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int G = 128;  // group size served by this path (one MFMA K)

// ---- fp8 e4m3 (OCP), round to nearest even; |a| <= 448 assumed ----------
__device__ inline uint32_t e4m3_rne(float v) {
  const uint32_t sign = v < 0.0f ? 0x80u : 0u;
  const float a = fabsf(v);
  if (a == 0.0f) return 0u;
  if (a < 0.015625f) {  // subnormal: q * 2^-9
    return sign | (uint32_t)rintf(a * 512.0f);  // q == 8 encodes 2^-6
  }
  int E;
  frexpf(a, &E);
  int e = E - 1;  // a in [2^e, 2^(e+1))
  float q = rintf((ldexpf(a, -e) - 1.0f) * 8.0f);
  if (q >= 8.0f) {
    q = 0.0f;
    e += 1;
  }
  int code = ((e + 7) << 3) | (int)q;
  code = code > 0x7e ? 0x7e : code;
  return sign | (uint32_t)code;
}

__device__ inline float e4m3_val(uint32_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  const float v = e == 0 ? ldexpf((float)m, -9) : ldexpf((float)(8 + m), e - 10);
  return (c & 0x80u) ? -v : v;
}

template <typename T>
__device__ inline float ld_act(const T* p);
template <>
__device__ inline float ld_act<float>(const float* p) { return *p; }
template <>
__device__ inline float ld_act<uint16_t>(const uint16_t* p) { return bf2f(*p); }

// Activation prep: one thread per (position, 32-column block).  Writes the
// hi/lo fp8 pieces in the B-operand lane order of the 16x16x128 MFMA
// (lane group q holds hardware k 16q..16q+15 and 64+16q..64+16q+15) and the
// E8M0 block scales.  Logical column 32q + 4n + d sits at hardware k
// 32q + 8d + n, matching the nibble order of the expanded plane words.
//   Xq [pos][K/128][piece][128] bytes, Xs [pos][K/128][piece][4] bytes
template <typename TIN>
__global__ void xprep_kernel(const TIN* __restrict__ in, int in_ld,
                             const int32_t* __restrict__ perm, int kdiv, int npos, int K,
                             uint8_t* __restrict__ Xq, uint8_t* __restrict__ Xs) {
  const int nb32 = K / 32;
  const int tid = blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= npos * nb32) return;
  const int pos = tid / nb32, kb = tid % nb32;
  const int g = kb >> 2, q = kb & 3, NG = K / G;
  const long row = perm ? (long)(perm[pos] / kdiv) : (long)pos;
  const TIN* src = in + row * in_ld + (long)kb * 32;
  float v[32];
  float amax = 0.0f;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    v[e] = ld_act<TIN>(src + e);
    amax = fmaxf(amax, fabsf(v[e]));
  }
  int s = 0;
  if (amax > 0.0f) {
    int E;
    frexpf(amax, &E);  // amax < 2^E  ->  amax / 2^(E-8) < 256
    s = E - 8;
    s = s < -120 ? -120 : (s > 120 ? 120 : s);
  }
  const size_t base = ((size_t)pos * NG + g) * 2;
  uint8_t* hi = Xq + base * 128;
  uint8_t* lo = hi + 128;
#pragma unroll
  for (int kl = 0; kl < 32; ++kl) {
    const int d = kl & 3, n = kl >> 2;
    const int khw = 32 * q + 8 * d + n;
    const int qq = khw < 64 ? (khw >> 4) : ((khw - 64) >> 4);
    const int ee = khw < 64 ? (khw & 15) : (16 + ((khw - 64) & 15));
    const float x = ldexpf(v[kl], -s);
    const uint32_t ch = e4m3_rne(x);
    const float r = x - e4m3_val(ch);
    const uint32_t cl = e4m3_rne(r * 16.0f);
    hi[qq * 32 + ee] = (uint8_t)ch;
    lo[qq * 32 + ee] = (uint8_t)cl;
  }
  Xs[base * 4 + q] = (uint8_t)(s + 127);
  Xs[(base + 1) * 4 + q] = (uint8_t)(s - 4 + 127);
}

__device__ inline v8i expand_sigma(uint32_t w) {
  v8i a;
  a[0] = (int)(((w << 3) & 0x88888888u) | 0x11111111u);
  a[1] = (int)(((w << 2) & 0x88888888u) | 0x11111111u);
  a[2] = (int)(((w << 1) & 0x88888888u) | 0x11111111u);
  a[3] = (int)((w & 0x88888888u) | 0x11111111u);
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

// fp4 code of (z - 1.5) replicated over a dword: z = 0..3 -> B, 9, 1, 3
__device__ inline v8i zero_operand(uint32_t z) {
  const uint32_t c = (0x319Bu >> (z << 2)) & 0xFu;
  const uint32_t dw = c * 0x11111111u;
  v8i a;
  a[0] = a[1] = a[2] = a[3] = (int)dw;
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

__device__ inline v4f mfma_fp4_fp8(const v8i& a, const v8i& b, v4f c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 4, 0, 0, sa, 0, sb);
}

__device__ inline float silu(float a) { return a / (1.0f + __expf(-a)); }

// elist[4*i]: expert, first position, end position, largest bit-width
template <bool SWIGLU, int NW>
__global__ __launch_bounds__(64 * NW) void decode_kernel(
    MwqView W, const int32_t* __restrict__ elist, const int32_t* __restrict__ ecount,
    const int32_t* __restrict__ perm, const uint8_t* __restrict__ topk_bits,
    const uint8_t* __restrict__ Xq, const uint8_t* __restrict__ Xs, int f,
    float* __restrict__ out, int out_ld) {
  __shared__ float red[NW][64][16];
  const int ei = blockIdx.y;
  if (ei >= *ecount) return;
  const int e = elist[4 * ei], p0 = elist[4 * ei + 1], p1 = elist[4 * ei + 2];
  const int mb = elist[4 * ei + 3];
  const int rb = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, j = lane & 15, piece = lane & 1;
  const int NG = W.cols / G;
  const int g0 = wave * NG / NW, g1 = (wave + 1) * NG / NW;
  const int ncol = p1 - p0;
  const int ncb = ncol > 8 ? 2 : 1;

  int posj[2], bitj[2];
  bool validj[2];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int t = cb * 8 + (j >> 1);
    validj[cb] = t < ncol;
    posj[cb] = p0 + t;
    bitj[cb] = validj[cb] ? (int)topk_bits[perm[posj[cb]]] : 0;
  }

  constexpr int NR = SWIGLU ? 2 : 1;
  v4f acc[NR][2];
#pragma unroll
  for (int rr = 0; rr < NR; ++rr)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) acc[rr][cb] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int g = g0; g < g1; ++g) {
    v8i bop[2];
    int bsc[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      bsc[cb] = 127;
      bop[cb] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
      if (cb < ncb && validj[cb]) {
        const size_t base = ((size_t)posj[cb] * NG + g) * 2 + piece;
        const uint4* src = (const uint4*)(Xq + base * 128 + q * 32);
        const uint4 u0 = src[0], u1 = src[1];
        bop[cb] = v8i{(int)u0.x, (int)u0.y, (int)u0.z, (int)u0.w,
                      (int)u1.x, (int)u1.y, (int)u1.z, (int)u1.w};
        bsc[cb] = Xs[base * 4 + q];
      }
    }
#pragma unroll
    for (int rr = 0; rr < NR; ++rr) {
      const int rowblock = rr == 0 ? rb : rb + f / 16;
      const size_t blk = W.block(e, rowblock, g);
      const uint32_t z = W.zeros[W.zero_idx(blk, j)];
      const uint2 s1 = *(const uint2*)(W.scales + W.scale_idx(blk, 0, 4 * q));
      const uint32_t w0 = W.planes[W.plane_word(blk, 0, lane)];
      const uint32_t w1 = W.planes[W.plane_word(blk, 1, lane)];
      const v8i a0 = expand_sigma(w0), a1 = expand_sigma(w1), au = zero_operand(z);
      const float sc[4] = {h2f((uint16_t)(s1.x & 0xffff)), h2f((uint16_t)(s1.x >> 16)),
                           h2f((uint16_t)(s1.y & 0xffff)), h2f((uint16_t)(s1.y >> 16))};
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        if (cb >= ncb) continue;
        v4f d = v4f{0.f, 0.f, 0.f, 0.f};
        d = mfma_fp4_fp8(a0, bop[cb], d, 127, bsc[cb]);
        d = mfma_fp4_fp8(a1, bop[cb], d, 128, bsc[cb]);
        d = mfma_fp4_fp8(au, bop[cb], d, 127, bsc[cb]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[rr][cb][r] = fmaf(-sc[r], d[r], acc[rr][cb][r]);
      }
      for (int p = 2; p < mb; ++p) {
        const uint32_t wp = W.planes[W.plane_word(blk, p, lane)];
        const uint2 sp2 = *(const uint2*)(W.scales + W.scale_idx(blk, p - 1, 4 * q));
        const v8i ap = expand_sigma(wp);
        const float sp[4] = {h2f((uint16_t)(sp2.x & 0xffff)), h2f((uint16_t)(sp2.x >> 16)),
                             h2f((uint16_t)(sp2.y & 0xffff)), h2f((uint16_t)(sp2.y >> 16))};
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          if (cb >= ncb) continue;
          const v4f d = mfma_fp4_fp8(ap, bop[cb], v4f{0.f, 0.f, 0.f, 0.f}, 128, bsc[cb]);
          if (p < bitj[cb]) {
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[rr][cb][r] = fmaf(-sp[r], d[r], acc[rr][cb][r]);
          }
        }
      }
    }
  }

  // reduce the groups split over the waves
#pragma unroll
  for (int rr = 0; rr < NR; ++rr)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][lane][rr * 8 + cb * 4 + r] = acc[rr][cb][r];
  __syncthreads();
  if (wave != 0) return;
  float v[NR][2][4];
#pragma unroll
  for (int rr = 0; rr < NR; ++rr)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float s = 0.0f;
        for (int w = 0; w < NW; ++w) s += red[w][lane][rr * 8 + cb * 4 + r];
        v[rr][cb][r] = s + __shfl_xor(s, 1, 64);  // hi + lo pieces
      }
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    if (cb >= ncb || !validj[cb] || piece != 0) continue;
    float* dst = out + (size_t)posj[cb] * out_ld + rb * 16 + 4 * q;
    float o[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = SWIGLU ? silu(v[0][cb][r]) * v[NR - 1][cb][r] : v[0][cb][r];
    *(float4*)dst = float4{o[0], o[1], o[2], o[3]};
  }
}

// Active-expert list for the decode kernels (ascending expert id).
__global__ void expert_list_kernel(const int32_t* __restrict__ offsets,
                                   const uint8_t* __restrict__ maxbit, int E, int L,
                                   int32_t* __restrict__ elist, int32_t* __restrict__ ecount) {
  if (threadIdx.x != 0) return;
  int n = 0;
  for (int e = 0; e < E; ++e) {
    if (maxbit[e] == 0) continue;
    elist[4 * n] = e;
    elist[4 * n + 1] = offsets[e * L];
    elist[4 * n + 2] = offsets[e * L + L];
    elist[4 * n + 3] = maxbit[e];
    ++n;
  }
  *ecount = n;
}

template <typename TIN>
hipError_t run_xprep(const TIN* in, int in_ld, const int32_t* perm, int kdiv, int npos, int K,
                     uint8_t* Xq, uint8_t* Xs, hipStream_t s) {
  const int n = npos * (K / 32);
  xprep_kernel<TIN><<<(n + 255) / 256, 256, 0, s>>>(in, in_ld, perm, kdiv, npos, K, Xq, Xs);
  return hipGetLastError();
}

}  // namespace

bool decode_path_ok(const d2moe_mwq* w13, const d2moe_mwq* w2, int T) {
  return T <= kDecodeMaxTokens && w13->group == 128 && w2->group == 128 && w13->b_min == 2 &&
         w2->b_min == 2;
}

hipError_t launch_decode_ffn(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                             const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                             const DecodeBuffers& b, hipStream_t s, const hipEvent_t* events) {
  hipError_t err;
  const int L = w13->b_max - w13->b_min + 1;
  const int npos = T * k;
  expert_list_kernel<<<1, 64, 0, s>>>(r->offsets, r->expert_maxbit, E, L, b.elist, b.ecount);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if (xd == D2MOE_BF16)
    err = run_xprep<uint16_t>((const uint16_t*)x, d, r->perm, k, npos, d, b.xq13, b.xs13, s);
  else
    err = run_xprep<float>((const float*)x, d, r->perm, k, npos, d, b.xq13, b.xs13, s);
  if (err != hipSuccess) return err;
  const int ny = E < npos ? E : npos;
  const MwqView W13 = view_of(w13), W2 = view_of(w2);
  if (events && (err = hipEventRecord(events[0], s)) != hipSuccess) return err;
  decode_kernel<true, 4><<<dim3(d_ff / 16, ny), 256, 0, s>>>(
      W13, b.elist, b.ecount, r->perm, r->topk_bits, b.xq13, b.xs13, d_ff, b.h32, d_ff);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if (events && (err = hipEventRecord(events[1], s)) != hipSuccess) return err;
  err = run_xprep<float>(b.h32, d_ff, nullptr, 1, npos, d_ff, b.xq2, b.xs2, s);
  if (err != hipSuccess) return err;
  if (events && (err = hipEventRecord(events[2], s)) != hipSuccess) return err;
  decode_kernel<false, 8><<<dim3(d / 16, ny), 512, 0, s>>>(
      W2, b.elist, b.ecount, r->perm, r->topk_bits, b.xq2, b.xs2, 0, b.y, d);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  if (events && (err = hipEventRecord(events[3], s)) != hipSuccess) return err;
  return hipSuccess;
}

}  // namespace d2moe
