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
// -s_b * D (A scale 2).  The base code Q (b_min planes) folds into chained
// MFMAs with A scales 2^p; at b_min = 2 a constant fp4 operand z - 1.5 joins
// the chain, so (Q - z) . x = -D as well (larger b_min: one more MFMA with an
// all-ones operand gives the activation sum for the zero-point term).  The
// first two base planes share one operand (values +-1/2, +-3/2).  Every
// residual plane thus costs one MFMA and one fp16-scaled FMA per output, and
// no weight is ever materialised as a number.  Tokens whose bit-width is below a plane get
// a zero coefficient for it; they share the loads.
//
// Work split: W1/W3 (decode13_kernel) gives each 16-row block of one active
// expert to two waves, each of which streams the W1 block and the matching
// W3 block of half the reduction dimension in alternate ring stages (so that
// a and c of the same outputs meet in its lanes); W2 gives each pair of
// adjacent 16-row blocks to four waves that stream both blocks of a quarter
// of the reduction (decode13_kernel) or, for small grids, each 16-row block
// to a 4-wave workgroup whose waves split the reduction (decode_kernel).
// Split waves reduce through LDS.  Requirement: group
// 128 (any nest start b_min).  An expert's positions are cut into work items
// of at most 8 or 16, each of which streams the expert's planes; the forward
// takes this path up to 64 tokens.
#include "internal.h"

#include <hip/hip_ext.h>

namespace d2moe {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int G = 128;  // group size served by this path (one MFMA K)
// A decode work item covers at most kDecodeCols tokens: the 16 MFMA columns
// hold each token's hi and lo activation pieces.
constexpr int kDecodeCols = 8;

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

// Activation prep (xprep_kernel below).  Each row is scaled by one
// power of two 2^s, with s taken from its largest magnitude so that
// |x| / 2^s < 256, and split into two fp8 e4m3 pieces, hi = rne(x / 2^s) and
// lo = rne(16 (x / 2^s - hi)).  Together they hold a bf16 value exactly
// while hi is a normal e4m3 number; smaller elements keep an absolute error
// below 2^-22 of the row maximum.  The pieces are written in the B-operand
// lane order of the 16x16x128 MFMA (lane group q holds hardware k
// 16q..16q+15 and 64+16q..64+16q+15); logical column 32q + 4n + d sits at
// hardware k 32q + 8d + n, matching the nibble order of the expanded plane
// words.  The position's info word Xs holds the E8M0 codes of 2^s (hi) and
// 2^(s-4) (lo) next to its token's bit-width.
//   Xq [pos][K/128][piece][128] bytes, Xs [pos] 32-bit words
// Position npos is an all-zero slot that decode lanes without a token read,
// so that every load in the decode loop is unconditional.
constexpr int kPrepThreads = 256;
constexpr int kPrepCols = 2048;  // columns per workgroup (16 groups)

__device__ inline int row_scale_exp(float amax) {
  int s = 0;
  if (amax > 0.0f) {
    int E;
    frexpf(amax, &E);  // amax < 2^E  ->  amax / 2^(E-8) < 256
    s = E - 8;
    s = s < -120 ? -120 : (s > 120 ? 120 : s);
  }
  return s;
}

// Grid (position, column slice of kPrepCols).  Every workgroup of a row
// takes the row's largest magnitude (from `rowmax`, or computed from the
// row, which is small and cached), then converts its slice, four output
// bytes per thread per step: output bytes 4j..4j+3 of a 16-byte run hold
// hardware k = 4j..4j+3, i.e. logical columns 32q + 4n + d for
// n = 4j'..4j'+3 (fixed d), so each thread reads four columns at stride 4 and
// stores one dword per piece.  The zero-slot workgroup of slice 0 also writes
// the work list of the decode kernels when `elist` is given: each active
// expert's positions in runs of at most `item` (experts widest first),
// elist[4 i] = expert,
// first position, end position, the expert's largest bit-width, and entries
// with bit-width 0 (no work) up to `nitems`, the grid's work-item count, so
// that a decode workgroup needs one load to learn its work.
template <typename TIN>
__device__ inline float row_absmax(const TIN* row, int K);
template <>
// Two 16-byte loads per thread in flight per round (a 4096-wide bf16 row is
// one round); the maximum does not depend on the order.
__device__ inline float row_absmax<uint16_t>(const uint16_t* row, int K) {
  float m = 0.0f;
  for (int c0 = 8 * threadIdx.x; c0 < K; c0 += 16 * kPrepThreads) {
    uint4 u[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = c0 + 8 * kPrepThreads * j;
      u[j] = c < K ? *(const uint4*)(row + c) : uint4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t w[4] = {u[j].x, u[j].y, u[j].z, u[j].w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        m = fmaxf(m, fmaxf(fabsf(bf2f((uint16_t)(w[i] & 0xffff))),
                           fabsf(bf2f((uint16_t)(w[i] >> 16)))));
    }
  }
  return m;
}
template <>
__device__ inline float row_absmax<float>(const float* row, int K) {
  float m = 0.0f;
  for (int c0 = 4 * threadIdx.x; c0 < K; c0 += 8 * kPrepThreads) {
    float4 v[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = c0 + 4 * kPrepThreads * j;
      v[j] = c < K ? *(const float4*)(row + c) : float4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v[j].x), fabsf(v[j].y)), fmaxf(fabsf(v[j].z), fabsf(v[j].w))));
  }
  return m;
}

// rowmax: partial maxima of |value| of each position's row as binary32 bits,
// rowmax[pos * rowmax_parts + i] (written by the producer of the rows, one
// entry per producing workgroup, so that no two producers update the same
// word), or NULL to compute the maximum here with 16-byte loads (rows are
// K % 128 == 0 elements on 16-byte aligned bases).
// Xs[pos] is the position's info word for the decode kernels: its token's
// bit-width (0 for the zero slot) in bits 0-7 and the E8M0 codes of the hi
// and lo activation pieces in bits 8-15 and 16-23.  Xs has 2 kDecodeCols - 1
// entries of padding past the zero slot, so a decode workgroup can read the
// words of 2 kDecodeCols positions from any first position.  bperm / tbits
// give the bit-width of position p as tbits[bperm[p]].
template <typename TIN>
__global__ __launch_bounds__(kPrepThreads) void xprep_kernel(
    const TIN* __restrict__ in, int in_ld, const int32_t* __restrict__ perm, int kdiv, int npos,
    int K, const uint32_t* __restrict__ rowmax, int rowmax_parts, uint8_t* __restrict__ Xq,
    uint32_t* __restrict__ Xs, const int32_t* __restrict__ bperm,
    const uint8_t* __restrict__ tbits, const int32_t* __restrict__ offsets,
    const uint8_t* __restrict__ maxbit, int E, int L, int32_t* __restrict__ elist, int nitems,
    int item) {
  __shared__ float wmax[kPrepThreads / 64];
  __shared__ int e_mb[64], e_lo[64], e_hi[64], e_cnt[64];  // per expert (E <= 64)
  const int pos = blockIdx.x, NG = K / G;
  if (pos == npos && blockIdx.y == 0 && elist) {  // workgroup-uniform
    // experts in order of their largest bit-width, widest first (then by
    // index), so that the longest work items are dispatched first and the
    // short ones fill the end of the grid.  One thread per expert: its rank
    // in that order gives its first slot.
    const int tid = threadIdx.x;
    if (tid < E) {
      const int mb = maxbit[tid], lo = offsets[tid * L], hi = offsets[tid * L + L];
      e_mb[tid] = mb;
      e_lo[tid] = lo;
      e_hi[tid] = hi;
      e_cnt[tid] = mb >= 1 && mb <= 8 ? (hi - lo + item - 1) / item : 0;
    }
    __syncthreads();
    int total = 0;
    for (int e = 0; e < E; ++e) total += e_cnt[e];
    if (tid < E && e_cnt[tid] > 0) {
      const int mb = e_mb[tid], hi = e_hi[tid];
      int n = 0;
      for (int e = 0; e < E; ++e)
        if (e_mb[e] > mb || (e_mb[e] == mb && e < tid)) n += e_cnt[e];
      for (int p = e_lo[tid]; p < hi; p += item, ++n) {
        elist[4 * n] = tid;
        elist[4 * n + 1] = p;
        elist[4 * n + 2] = min(p + item, hi);
        elist[4 * n + 3] = mb;
      }
    }
    // the remaining slots of the grid get no work (largest bit-width 0)
    for (int n = total + tid; n < nitems; n += kPrepThreads)
      elist[4 * n] = elist[4 * n + 1] = elist[4 * n + 2] = elist[4 * n + 3] = 0;
  }
  const TIN* src = nullptr;
  if (pos < npos) src = in + (long)(perm ? perm[pos] / kdiv : pos) * in_ld;
  float amax = 0.0f;
  if (src) {
    if (rowmax) {
      // four words per thread in flight per round (896 per row at the
      // Mixtral width: one round), not one dependent load per step
      const uint32_t* rm = rowmax + (size_t)pos * rowmax_parts;
      for (int i0 = threadIdx.x; i0 < rowmax_parts; i0 += 4 * kPrepThreads) {
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = i0 + j * kPrepThreads;
          v[j] = i < rowmax_parts ? __uint_as_float(rm[i]) : 0.0f;
        }
        amax = fmaxf(amax, fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])));
      }
    } else {
      amax = row_absmax<TIN>(src, K);
    }
  }
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = 0.0f;
  for (int w = 0; w < kPrepThreads / 64; ++w) amax = fmaxf(amax, wmax[w]);
  const int s = row_scale_exp(amax);
  uint32_t* row = (uint32_t*)(Xq + (size_t)pos * NG * 256);
  const int c0 = blockIdx.y * kPrepCols, c1 = min(K, c0 + kPrepCols);
  // one dword per thread per step: output dword u of the row covers
  // group u / 64, piece 0 (hi) dwords 0..31 of the group's 64.  Two steps
  // per round, both steps' loads issued before either converts (a slice of
  // 2048 columns is one round).
  constexpr int kSteps = 2;
  for (int u0 = c0 / 4 + threadIdx.x; u0 < c1 / 4; u0 += kSteps * kPrepThreads) {
    float xv[kSteps][4];
#pragma unroll
    for (int j = 0; j < kSteps; ++j) {
      const int u = u0 + j * kPrepThreads;
      const int g = u >> 5, w = u & 31;                 // hi dword w of group g
      const int qq = w >> 3, e4 = (w & 7) * 4;          // lane group, first byte
      const int khw = e4 < 16 ? 16 * qq + e4 : 64 + 16 * qq + (e4 - 16);
      const int kb = khw >> 5, dd = (khw & 31) >> 3, n0 = khw & 7;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int col = g * G + 32 * kb + 4 * (n0 + i) + dd;
        xv[j][i] = src && u < c1 / 4 ? ld_act<TIN>(src + col) : 0.0f;
      }
    }
#pragma unroll
    for (int j = 0; j < kSteps; ++j) {
      const int u = u0 + j * kPrepThreads;
      if (u < c1 / 4) {
        const int g = u >> 5, w = u & 31;
        uint32_t hi = 0, lo = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = ldexpf(xv[j][i], -s);
          const uint32_t ch = e4m3_rne(x);
          const float r = x - e4m3_val(ch);
          const uint32_t cl = e4m3_rne(r * 16.0f);
          hi |= ch << (8 * i);
          lo |= cl << (8 * i);
        }
        row[g * 64 + w] = hi;
        row[g * 64 + 32 + w] = lo;
      }
    }
  }
  if (threadIdx.x == 0 && blockIdx.y == 0) {
    const uint32_t bits = pos < npos ? tbits[bperm[pos]] : 0u;
    Xs[pos] = bits | ((uint32_t)(s + 127) << 8) | ((uint32_t)(s - 4 + 127) << 16);
  }
}

// Opaque copies of the two masks used by expand_sigma: held in VGPRs, they
// let each output dword be one shift plus one v_and_or_b32 (the three-operand
// form takes no literal on this target).
struct SigmaConsts {
  uint32_t m8, c1;
};
__device__ inline SigmaConsts sigma_consts() {
  SigmaConsts k;
  asm volatile("" : "=v"(k.m8) : "0"(0x88888888u));
  asm volatile("" : "=v"(k.c1) : "0"(0x11111111u));
  return k;
}

// fp4 e2m1 operand of one plane word: bit 4n+d of w becomes the sign of
// nibble n of dword d, magnitude 0.5, so a set bit reads as -0.5.
__device__ inline v8i expand_sigma(uint32_t w, const SigmaConsts& k) {
  v8i a;
  a[0] = (int)(((w << 3) & k.m8) | k.c1);
  a[1] = (int)(((w << 2) & k.m8) | k.c1);
  a[2] = (int)(((w << 1) & k.m8) | k.c1);
  a[3] = (int)((w & k.m8) | k.c1);
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

// fp4 e2m1 operand of the first two planes of the base code together: the
// weight with bit b0 in plane 0 and b1 in plane 1 reads 3/2 - (b0 + 2 b1),
// one of +-1/2, +-3/2 (sign b1; the exponent bit of value 1 set when
// b0 == b1; mantissa bit 1), in the nibble order of expand_sigma.
__device__ inline v8i expand_pair(uint32_t w0, uint32_t w1, const SigmaConsts& k) {
  const uint32_t e = ~(w0 ^ w1);
  constexpr uint32_t m2 = 0x22222222u;
  v8i a;
  a[0] = (int)((((w1 << 3) & k.m8) | k.c1) | ((e << 1) & m2));
  a[1] = (int)((((w1 << 2) & k.m8) | k.c1) | (e & m2));
  a[2] = (int)((((w1 << 1) & k.m8) | k.c1) | ((e >> 1) & m2));
  a[3] = (int)(((w1 & k.m8) | k.c1) | ((e >> 2) & m2));
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

// Cross-lane product: every call sits in wave-uniform control flow (no
// per-lane condition guards an MFMA or the use of its result in this file;
// per-token predication is done through the activation block scale).
//
// This 8-pass MFMA must not write registers it is still reading, but the
// compiler treats a 4-register result as free to overlap the operands.  Each
// call therefore passes its result through an empty asm that also reads the
// operands: the asm must follow the MFMA (it consumes the result), and the
// operands are live up to it, so the result is always given registers of
// its own.  (An asm that only reads the operands is not enough: nothing
// orders it after the MFMA, and the scheduler may move it above.)
__device__ inline v4i lo4(const v8i& a) { return v4i{a[0], a[1], a[2], a[3]}; }

__device__ inline v4f mfma_fp4_fp8(const v8i& a, const v8i& b, int sa, int sb) {
  v4f d = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
      a, b, v4f{0.f, 0.f, 0.f, 0.f}, 4, 0, 0, sa, 0, sb);
  asm volatile("" : "+v"(d) : "v"(lo4(a)), "v"(b), "v"(sa), "v"(sb));
  return d;
}
__device__ inline v4f mfma_fp4_fp8(const v8i& a, const v8i& b, v4f c, int sa, int sb) {
  v4f d = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 4, 0, 0, sa, 0, sb);
  asm volatile("" : "+v"(d) : "v"(lo4(a)), "v"(b), "v"(c), "v"(sa), "v"(sb));
  return d;
}

__device__ inline float silu(float a) { return a / (1.0f + __expf(-a)); }

// Four binary16 scales (rows 4q..4q+3) as floats.
__device__ inline void scales4(uint2 s, float (&out)[4]) {
  out[0] = h2f((uint16_t)(s.x & 0xffff));
  out[1] = h2f((uint16_t)(s.x >> 16));
  out[2] = h2f((uint16_t)(s.y & 0xffff));
  out[3] = h2f((uint16_t)(s.y >> 16));
}

// Per-wave LDS ring for the weight stream.  One stage holds one group of the
// wave's 16 rows at MB planes of a nest that starts at BMIN bits, packed as
// [planes MB x 256 B][scales LV x 32 B][zero points 16 B] with
// LV = MB - BMIN + 1 scale levels, copied from global memory by the LDS DMA
// engine so that data in flight costs no registers.  Each DMA instruction
// moves 16 bytes per lane into consecutive LDS addresses; lane slot s of the
// stage (s = 64 i + lane for instruction i) fetches plane bytes for
// s < 16 MB, scale bytes for the next 2 LV slots and the zero points in the
// last one, each from its own array.
constexpr int kDepth = 4;               // stages: the DMA runs kDepth-1 groups ahead
constexpr int kCpolNT = 2;              // cache-policy operand of the DMA: nt

template <int MB, int BMIN>
struct StageLayout {
  static constexpr int levels = MB - BMIN + 1;
  static constexpr int scale_off = 256 * MB;
  static constexpr int zero_off = scale_off + 32 * levels;
  static constexpr int slots = 16 * MB + 2 * levels + 1;
  static constexpr int ops = (slots + 63) / 64;  // DMA instructions per group
};

// Bytes per stage: the largest stage of the nest (MB = 8), 2304 for
// BMIN >= 2 and 2320 for BMIN = 1.
template <int BMIN>
constexpr int stage_bytes() {
  return 16 * StageLayout<8, BMIN>::slots <= 2304 ? 2304 : 16 * StageLayout<8, BMIN>::slots;
}

#define D2MOE_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define D2MOE_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

// NCB column blocks of kDecodeCols tokens share every plane operand; block c
// holds the work item's positions 8 c .. 8 c + 7.
template <int NCB>
struct WaveCtx {
  const uint8_t* pl;   // plane words of group 0 of this row-block (bytes)
  const uint8_t* sc;   // scales of group 0 (bytes)
  const uint8_t* zp;   // zero points of group 0
  int pl_step, sc_step;  // bytes per group
  int lane, q, j;
  uint32_t info[NCB];      // position info words (bit-width, activation scale codes)
  int info_shift;          // bit offset of this lane's piece's scale code in `info`
  const uint8_t* xq[NCB];  // activation pieces of group 0, this lane
  uint64_t lmask[NCB];     // lanes holding a token (lane 0 always included)
  SigmaConsts k;
  uint32_t lds_pl, lds_sc, lds_z, lds_zq;  // this lane's LDS read bases in stage 0
};

// Source of each DMA instruction's 16 bytes for this lane: the address for
// group 0 and the stride per group (0 for lanes past the last slot, which
// do not issue).
template <int MB, int BMIN>
struct DmaPlan {
  const uint8_t* a0[StageLayout<MB, BMIN>::ops];
  int step[StageLayout<MB, BMIN>::ops];
};

template <int MB, int BMIN, typename Ctx>
__device__ inline DmaPlan<MB, BMIN> dma_plan(const Ctx& c) {
  using SL = StageLayout<MB, BMIN>;
  DmaPlan<MB, BMIN> d;
#pragma unroll
  for (int i = 0; i < SL::ops; ++i) {
    const int s = 64 * i + c.lane;
    if (s < 16 * MB) {
      d.a0[i] = c.pl + 16 * s;
      d.step[i] = c.pl_step;
    } else if (s < 16 * MB + 2 * SL::levels) {
      d.a0[i] = c.sc + 16 * (s - 16 * MB);
      d.step[i] = c.sc_step;
    } else if (s == SL::slots - 1) {
      d.a0[i] = c.zp;
      d.step[i] = 16;
    } else {
      d.a0[i] = c.pl;
      d.step[i] = 0;
    }
  }
  return d;
}

template <int MB, int BMIN, typename Ctx>
__device__ inline void dma_group(const DmaPlan<MB, BMIN>& d, const Ctx& c, int g, uint8_t* st) {
  using SL = StageLayout<MB, BMIN>;
#pragma unroll
  for (int i = 0; i < SL::ops; ++i) {
    // every instruction has lane 0 active (slot 64 i < slots), so each one
    // issues and is counted by vmcnt.  Plane words are read once per call, so
    // instructions that carry only plane words are marked nontemporal (cache
    // policy nt): streaming them past the caches reads HBM markedly faster on
    // this chip than default-policy loads.  Scales and zero points are short
    // runs that share cache lines with the next group's, so they keep the
    // default policy.
    if (64 * i + c.lane < SL::slots) {
      if (64 * (i + 1) <= 16 * MB)  // constant once the loop is unrolled
        __builtin_amdgcn_global_load_lds(D2MOE_GPTR(d.a0[i] + (size_t)g * d.step[i]),
                                         D2MOE_LPTR(st + 1024 * i), 16, 0, kCpolNT);
      else
        __builtin_amdgcn_global_load_lds(D2MOE_GPTR(d.a0[i] + (size_t)g * d.step[i]),
                                         D2MOE_LPTR(st + 1024 * i), 16, 0, 0);
    }
  }
}

template <int NCB>
struct BData {
  v4i lo[NCB], hi[NCB];  // this lane's 32 bytes of activation pieces per column block
};

// Activation loads are issued as inline assembly for the same reason as the
// ring reads: with LDS DMA in flight the compiler cannot tell which vector
// loads have completed and would wait for all of them (draining the weight
// prefetch) before the first use of these registers.  They are ordered by the
// explicit vmcnt waits of the group loop instead; ready_b() re-binds the
// registers after that wait so that no use can move above it.  The "memory"
// clobber keeps their issue order fixed relative to the DMA instructions,
// which the wait counts rely on.
// Only the lanes in `m` load (EXEC is narrowed and restored inside the asm);
// the other lanes keep `v`.  `m` always contains lane 0, so the instruction
// is always issued and counted by vmcnt.  s_and_saveexec writes SCC, which
// the compiler may otherwise keep live across the asm (for instance the carry
// between the two halves of a 64-bit scalar address add), hence the clobber.
__device__ inline void gload16(v4i& v, const uint8_t* p, uint64_t m) {
  uint64_t saved;
  asm volatile(
      "s_and_saveexec_b64 %1, %3\n\t"
      "global_load_dwordx4 %0, %2, off\n\t"
      "s_mov_b64 exec, %1"
      : "+v"(v), "=&s"(saved)
      : "v"(p), "s"(m)
      : "memory", "scc");
}

// Two memory instructions per live column block (the first NL), issued by the
// lanes that hold a token (lane 0 always does); the other lanes keep the zeros
// they were given before the loop.
template <int NL, int NCB>
__device__ inline void load_b(BData<NCB>& t, const WaveCtx<NCB>& c, int g) {
#pragma unroll
  for (int cb = 0; cb < NL; ++cb) {
    const uint8_t* src = c.xq[cb] + (size_t)g * 256;
    gload16(t.lo[cb], src, c.lmask[cb]);
    gload16(t.hi[cb], src + 16, c.lmask[cb]);
  }
}

// Called after the wait that covers the loads of `t`.
template <int NCB>
__device__ inline void ready_b(BData<NCB>& t) {
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) asm volatile("" : "+v"(t.lo[cb]), "+v"(t.hi[cb]));
}

template <int NCB>
__device__ inline v8i b8(const BData<NCB>& t, int cb) {
  return v8i{t.lo[cb][0], t.lo[cb][1], t.lo[cb][2], t.lo[cb][3],
             t.hi[cb][0], t.hi[cb][1], t.hi[cb][2], t.hi[cb][3]};
}

// LDS reads of a ring stage are issued as inline assembly: the compiler's
// wait insertion would otherwise treat every LDS read as possibly reading a
// DMA still in flight and drain all of them.  The explicit vmcnt wait before
// the stage is consumed (wait_vm) orders the DMA, and one lgkmcnt wait after
// the reads orders the reads; each value is then re-bound by an empty asm so
// no use can move above that wait.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
template <int OFF>
__device__ inline uint32_t lds_rd32(uint32_t a) {
  uint32_t v;
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF));
  return v;
}
template <int OFF>
__device__ inline uint2 lds_rd64(uint32_t a) {
  uint2 v;
  asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF));
  return v;
}
template <int OFF>
__device__ inline uint32_t lds_rdu8(uint32_t a) {
  uint32_t v;
  asm volatile("ds_read_u8 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF));
  return v;
}
template <int P, int MB, int SOFF>
struct PlaneReader {
  static __device__ inline void run(uint32_t a, uint32_t (&w)[MB]) {
    w[P] = lds_rd32<SOFF + P * 256>(a);
    PlaneReader<P + 1, MB, SOFF>::run(a, w);
  }
};
template <int MB, int SOFF>
struct PlaneReader<MB, MB, SOFF> {
  static __device__ inline void run(uint32_t, uint32_t (&)[MB]) {}
};
template <int L, int LV, int SOFF>
struct ScaleReader {
  static __device__ inline void run(uint32_t a, uint2 (&sc)[LV]) {
    sc[L] = lds_rd64<SOFF + L * 32>(a);
    ScaleReader<L + 1, LV, SOFF>::run(a, sc);
  }
};
template <int LV, int SOFF>
struct ScaleReader<LV, LV, SOFF> {
  static __device__ inline void run(uint32_t, uint2 (&)[LV]) {}
};

// Plane words, the four binary16 scales per level of the lane's output rows,
// and the zero point of the lane's operand row (BMIN <= 2) or the four zero
// points of its output rows (BMIN >= 3).
template <int MB, int BMIN, int SOFF, typename Ctx>
__device__ inline void read_stage(const Ctx& c, uint32_t (&w)[MB],
                                  uint2 (&sc)[StageLayout<MB, BMIN>::levels], uint32_t& z) {
  using SL = StageLayout<MB, BMIN>;
  PlaneReader<0, MB, SOFF>::run(c.lds_pl, w);
  ScaleReader<0, SL::levels, SOFF + SL::scale_off>::run(c.lds_sc, sc);
  if constexpr (BMIN <= 2)
    z = lds_rdu8<SOFF + SL::zero_off>(c.lds_z);
  else
    z = lds_rd32<SOFF + SL::zero_off>(c.lds_zq);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int p = 0; p < MB; ++p) asm volatile("" : "+v"(w[p]));
#pragma unroll
  for (int l = 0; l < SL::levels; ++l) asm volatile("" : "+v"(sc[l]));
  asm volatile("" : "+v"(z));
}

// fp4 operand of the constant z - (2^BMIN - 1)/2 for BMIN <= 2 (it is one of
// +-0.5, +-1.5): BMIN = 2, z = 0..3 -> B, 9, 1, 3; BMIN = 1, z = 0..1 -> 9, 1.
template <int BMIN>
__device__ inline v8i zero_operand(uint32_t z) {
  const uint32_t c = ((BMIN == 2 ? 0x319Bu : 0x19u) >> (z << 2)) & 0xFu;
  const uint32_t dw = c * 0x11111111u;
  v8i a;
  a[0] = a[1] = a[2] = a[3] = (int)dw;
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

// fp4 operand of all ones (code 2 is 1.0).
__device__ inline v8i ones_operand() {
  v8i a;
  a[0] = a[1] = a[2] = a[3] = 0x22222222;
  a[4] = a[5] = a[6] = a[7] = 0;
  return a;
}

// One group of the wave's 16 rows against the column blocks' activations.
//   Base level: plane p < BMIN with A scale 2^p reads 2^p (1/2 - bit p)
//   (planes 0 and 1 as one operand, 3/2 - (b0 + 2 b1)), so the chained
//   MFMAs give m = h S - Q.x with h = (2^BMIN - 1)/2 and S the column's
//   activation sum, and s1 (Q - z).x = -s1 m + s1 (h - z) S.  For
//   BMIN <= 2 the constant operand z - h joins the chain, leaving -s1 m; for
//   larger BMIN, S comes from one MFMA with an all-ones operand and the
//   second term is one FMA per output.
//   Residual level p >= BMIN: one MFMA with A scale 2 (-sigma) and one FMA
//   with -s_p.
// Planes a token does not request are switched off through its activation
// block scale: E8M0 code 0 scales that column's products by 2^-127, which
// leaves at most ~1e-33 (|x| < 2^9 per fp8 piece, 128 terms) in place of an
// exact zero.
template <int MB, int BMIN, int SOFF, int NL, int NCB>
__device__ inline void compute_group(const BData<NCB>& t, const WaveCtx<NCB>& c,
                                     v4f (&acc)[NCB]) {
  static_assert(NL >= 1 && NL <= NCB, "live column blocks");
  using SL = StageLayout<MB, BMIN>;
  int bit[NCB], bsc[NCB];
#pragma unroll
  for (int cb = 0; cb < NL; ++cb) {
    bit[cb] = (int)(c.info[cb] & 0xffu);                     // token's bit-width
    bsc[cb] = (int)((c.info[cb] >> c.info_shift) & 0xffu);   // its activation scale code
  }
  const SigmaConsts& k = c.k;
  uint32_t w[MB];
  uint2 sw[SL::levels];
  uint32_t z;
  read_stage<MB, BMIN, SOFF>(c, w, sw, z);
  float s1[4];
  scales4(sw[0], s1);
  float zc[4];  // s1 (h - z) of the lane's output rows (BMIN >= 3)
  if constexpr (BMIN >= 3) {
    constexpr float h = 0.5f * (float)((1 << BMIN) - 1);
#pragma unroll
    for (int r = 0; r < 4; ++r) zc[r] = s1[r] * (h - (float)((z >> (8 * r)) & 0xffu));
  }
  // base chain, one expanded operand at a time for all column blocks;
  // planes 0 and 1 share one operand (A scale 1), so a nest from 2 bits
  // chains the zero-point operand and the pair
  v4f m[NCB];
  if constexpr (BMIN <= 2) {
    const v8i au = zero_operand<BMIN>(z);
#pragma unroll
    for (int cb = 0; cb < NL; ++cb) m[cb] = mfma_fp4_fp8(au, b8(t, cb), 127, bsc[cb]);
    const v8i ap = BMIN == 2 ? expand_pair(w[0], w[BMIN - 1], k) : expand_sigma(w[0], k);
#pragma unroll
    for (int cb = 0; cb < NL; ++cb) m[cb] = mfma_fp4_fp8(ap, b8(t, cb), m[cb], 127, bsc[cb]);
  } else {
    const v8i a01 = expand_pair(w[0], w[1], k);
#pragma unroll
    for (int cb = 0; cb < NL; ++cb) m[cb] = mfma_fp4_fp8(a01, b8(t, cb), 127, bsc[cb]);
  }
#pragma unroll
  for (int p = 2; p < BMIN; ++p) {
    const v8i ap = expand_sigma(w[p], k);
#pragma unroll
    for (int cb = 0; cb < NL; ++cb) m[cb] = mfma_fp4_fp8(ap, b8(t, cb), m[cb], 127 + p, bsc[cb]);
  }
#pragma unroll
  for (int cb = 0; cb < NL; ++cb) {
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[cb][r] = fmaf(-s1[r], m[cb][r], acc[cb][r]);
    if constexpr (BMIN >= 3) {
      const v4f so = mfma_fp4_fp8(ones_operand(), b8(t, cb), 127, bsc[cb]);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[cb][r] = fmaf(zc[r], so[r], acc[cb][r]);
    }
  }
#pragma unroll
  for (int p = BMIN; p < MB; ++p) {
    const v8i ap = expand_sigma(w[p], k);
    float sp[4];
    scales4(sw[p - BMIN + 1], sp);
#pragma unroll
    for (int cb = 0; cb < NL; ++cb) {
      const int bs = p < bit[cb] ? bsc[cb] : 0;
      const v4f d = mfma_fp4_fp8(ap, b8(t, cb), 128, bs);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[cb][r] = fmaf(-sp[r], d[r], acc[cb][r]);
    }
  }
}

// Wait until at most N memory instructions of this wave are outstanding, and
// keep every later LDS read below the wait.
template <int N>
__device__ inline void wait_vm() {
  if constexpr (N == 0)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// One wave's share: groups [g0, g1) at MB planes of a nest starting at BMIN
// bits, through this wave's ring of kDepth stages (stage_bytes<BMIN>() bytes
// apart, starting at `ring`).  Order of issue:
// the prologue sends the DMA of g0 and g0+1, the activations of g0, then the
// DMA of g0+2; the step that computes group g sends the activations of g+1
// and the DMA of g+3, then waits.  Before that wait, the memory instructions
// issued after the activations of g are the DMA of g+2, the activations of
// g+1 and the DMA of g+3 (those that exist), and every earlier one covers
// group g; vector-memory instructions of a wave complete in order, so
// waiting until only those remain outstanding makes the stage and the
// activations of g ready.  The DMA of g+3 overwrites the stage of g-1, whose
// LDS reads completed in the previous step.  The loop is unrolled by kDepth
// so every stage offset is a constant; the steps past the end are skipped by
// guards rather than left by `break`, so the loop has one exit and the
// compiler adds no exit flag that carries undefined loop values.  NL: the
// column blocks that hold positions (the first NL of NCB).
template <int MB, int BMIN, int NL, int NCB>
__device__ inline void decode_groups(const WaveCtx<NCB>& c, uint8_t* ring, int g0, int g1,
                                     v4f (&acc)[NCB]) {
  static_assert(kDepth == 4, "the unrolled step below assumes four stages");
  if (g0 >= g1) return;
  constexpr int ND = StageLayout<MB, BMIN>::ops, NB = 2 * NL;
  constexpr int kStage = stage_bytes<BMIN>();
  const DmaPlan<MB, BMIN> plan = dma_plan<MB, BMIN>(c);
  BData<NCB> B[2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) B[i].lo[cb] = B[i].hi[cb] = v4i{0, 0, 0, 0};
  dma_group<MB, BMIN>(plan, c, g0, ring);
  if (g0 + 1 < g1) dma_group<MB, BMIN>(plan, c, g0 + 1, ring + kStage);
  load_b<NL>(B[0], c, g0);
  if (g0 + 2 < g1) dma_group<MB, BMIN>(plan, c, g0 + 2, ring + 2 * kStage);
#define D2MOE_STEP(K)                                                        \
  if (g + (K) < g1) {                                                        \
    const int gg = g + (K);                                                  \
    if (gg + 1 < g1) load_b<NL>(B[((K) + 1) & 1], c, gg + 1);                \
    if (gg + 3 < g1) {                                                       \
      dma_group<MB, BMIN>(plan, c, gg + 3, ring + (((K) + 3) % kDepth) * kStage); \
      wait_vm<2 * ND + NB>();                                                \
    } else if (gg + 2 < g1) {                                                \
      wait_vm<ND + NB>();                                                    \
    } else if (gg + 1 < g1) {                                                \
      wait_vm<NB>();                                                         \
    } else {                                                                 \
      wait_vm<0>();                                                          \
    }                                                                        \
    ready_b(B[(K) & 1]);                                                     \
    compute_group<MB, BMIN, ((K) % kDepth) * kStage, NL>(B[(K) & 1], c, acc); \
  }
  for (int g = g0; g < g1; g += kDepth) {
    D2MOE_STEP(0)
    D2MOE_STEP(1)
    D2MOE_STEP(2)
    D2MOE_STEP(3)
  }
#undef D2MOE_STEP
  wait_vm<0>();  // as in decode_pairs: explicit on every exit edge of the loop
}


// elist[4*i]: expert, first position, end position (at most NCB * kDecodeCols
// positions), largest bit-width of the expert (0: no work).  Xs: position
// info words (bit-width, activation scale codes) from the activation prep,
// padded so that NCB * kDecodeCols words can be read from any position.
// One W2 row block per workgroup: its NW waves split the groups and combine
// their partial sums through LDS (each wave's partial sums go to its own
// ring, which is idle by then).  NCB column blocks of 8 tokens share every
// plane operand (two when experts hold more than 4 positions on average,
// three above 12), at 4 waves per SIMD for one block, 3 for two and 2 for
// three (three blocks need more than the 168 registers of 3 waves).
template <int NW, int NCB, int BMIN>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(NCB == 1 ? 4 : NCB == 2 ? 3 : 2)))
void decode_kernel(MwqView W, const int32_t* __restrict__ elist, const uint8_t* __restrict__ Xq,
                   const uint32_t* __restrict__ Xs, int npos, float* __restrict__ out,
                   int out_ld) {
  constexpr int kStage = stage_bytes<BMIN>();
  __shared__ __attribute__((aligned(16))) uint8_t ring[NW][kDepth * kStage];
  static_assert(kDepth * kStage >= NCB * 64 * 4 * (int)sizeof(float),
                "partial sums fit the ring");
  const int ei = blockIdx.y;
  const int e = elist[4 * ei], p0 = elist[4 * ei + 1], p1 = elist[4 * ei + 2];
  const int mb_req = elist[4 * ei + 3];
  if (mb_req == 0) return;
  // planes actually read never exceed the packed nest, whatever the routing
  const int mb = mb_req < W.b_max ? mb_req : W.b_max;
  const int rb = blockIdx.x;
  const int lane = threadIdx.x & 63;
  // wave-uniform by construction; readfirstlane lets the compiler keep the
  // group loop in scalar control flow
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int NG = W.cols / G;
  constexpr int KS = NW;  // waves splitting the groups
  const int wk = wave;
  const int g0 = wk * NG / KS, g1 = (wk + 1) * NG / KS;
  const int ncol = p1 - p0;

  WaveCtx<NCB> c;
  c.lane = lane;
  c.q = lane >> 4;
  c.j = lane & 15;
  const int piece = lane & 1;
  const int t = c.j >> 1;
  c.info_shift = 8 + 8 * piece;
  bool valid[NCB];
  int pos[NCB];
  {
    // the info words of the item's positions are wave-uniform reads (scalar
    // cache, ordered by lgkmcnt), so waiting for them never holds back the
    // weight DMA; each lane then picks its token's word
    uint32_t iw[NCB * kDecodeCols];
#pragma unroll
    for (int i = 0; i < NCB * kDecodeCols; ++i) iw[i] = Xs[p0 + i];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const int tc = kDecodeCols * cb + t;
      valid[cb] = tc < ncol;
      pos[cb] = p0 + tc;
      const int src = valid[cb] ? pos[cb] : npos;  // zero slot when no token
      const size_t base = ((size_t)src * NG) * 2 + piece;  // group 0
      c.xq[cb] = Xq + base * 128 + c.q * 32;
      // lane 0 always loads (its own slot or the zero slot), so that every
      // activation load instruction issues and is counted by vmcnt
      c.lmask[cb] = __ballot(valid[cb]) | 1ull;
      uint32_t info = 0u;
#pragma unroll
      for (int i = 0; i < kDecodeCols; ++i) info = t == i ? iw[kDecodeCols * cb + i] : info;
      c.info[cb] = valid[cb] ? info : 0u;  // no token: bit-width 0, zero activations
    }
  }

  const size_t blk0 = W.block(e, rb, 0);
  c.pl = (const uint8_t*)(W.planes + W.plane_word(blk0, 0, 0));
  c.sc = (const uint8_t*)(W.scales + W.scale_idx(blk0, 0, 0));
  c.zp = W.zeros + W.zero_idx(blk0, 0);
  c.pl_step = W.b_max * 64 * 4;
  c.sc_step = W.levels() * 16 * 2;
  c.k = sigma_consts();
  {
    const uint32_t base = lds_addr(ring[wave]);
    c.lds_pl = base + 4 * lane;
    c.lds_sc = base + 8 * c.q;
    c.lds_z = base + c.j;
    c.lds_zq = base + 4 * c.q;
  }

  v4f acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = v4f{0.f, 0.f, 0.f, 0.f};
  // column blocks past the item's last position are skipped: with more
  // than one block, the item's block count picks the group loop (three-block
  // kernels serve items of two or three, two-block kernels of one or two)
  const bool full = ncol > kDecodeCols * (NCB - 1);
  switch (mb) {
#define D2MOE_CASE(MB)                                                                   \
  case MB:                                                                               \
    if constexpr (MB >= BMIN) {                                                          \
      if (full || NCB == 1)                                                              \
        decode_groups<MB, BMIN, NCB>(c, ring[wave], g0, g1, acc);                        \
      else                                                                               \
        decode_groups<MB, BMIN, NCB == 1 ? 1 : NCB - 1>(c, ring[wave], g0, g1, acc);     \
    }                                                                                    \
    break;
    D2MOE_CASE(1) D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6)
    D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
    default: break;
  }

  // every DMA of this wave has completed (the last step waits for all), so
  // its ring can hold its partial sums
  float4* red = (float4*)ring[wave];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
    red[64 * cb + lane] = float4{acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]};
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    float4 sum = float4{0.f, 0.f, 0.f, 0.f};
    for (int w = 0; w < KS; ++w) {
      const float4 part = ((const float4*)ring[w])[64 * cb + lane];
      sum.x += part.x; sum.y += part.y; sum.z += part.z; sum.w += part.w;
    }
    const float o0 = sum.x + __shfl_xor(sum.x, 1, 64);  // hi + lo pieces
    const float o1 = sum.y + __shfl_xor(sum.y, 1, 64);
    const float o2 = sum.z + __shfl_xor(sum.z, 1, 64);
    const float o3 = sum.w + __shfl_xor(sum.w, 1, 64);
    if (valid[cb] && piece == 0)
      *(float4*)(out + (size_t)pos[cb] * out_ld + rb * 16 + 4 * c.q) = float4{o0, o1, o2, o3};
  }
}

// ---- paired-block kernels: each wave streams two weight blocks in turn
//
// A wave streams two 16-row blocks over its share of the reduction
// dimension, one group of each in turn: ring stage s holds group s / 2 of the
// first block (s even) or of the second (s odd).  One activation load serves
// both stages of a group.  For W1/W3 the two blocks are the W1 block and the
// matching W3 block, so each lane ends with a and c of the same outputs; for
// W2 they are two adjacent row blocks.
//
// Order of issue: the prologue sends the DMA of stage 0, the activations of
// group 0, then the DMA of stages 1 and 2; the step that computes stage s
// sends the activations of group s/2 + 1 (even s) and the DMA of stage s + 3,
// then waits.  In issue order the newest instructions needed by stage s are
// the activations of its group (even s) or its own DMA (odd s); in both cases
// exactly the DMA of stages s+1..s+3 and the activations of group s/2 + 1
// (those that exist) were issued after them, and vector-memory instructions
// of a wave complete in order, so waiting until only those remain
// outstanding makes the stage and its activations ready.  The DMA of stage
// s + 3 overwrites the stage of s - 1, whose LDS reads completed in the
// previous step.  The loop is unrolled by kDepth stages (two groups) so that
// every ring offset and activation buffer index is a constant, with guards
// on the steps past the end as in decode_groups.
// DMA of one stage.  Instructions that carry only plane words address them
// from the wave-uniform base of group g's planes (16 bytes per lane, 1 KB per
// instruction), so they hold no per-lane pointer.  The last, mixed
// instruction (scales and zero points, and plane words when the nest is not
// a multiple of four planes) keeps a per-lane source pointer, stride and
// second-block offset (MixedDma).  `W3` selects the second block.
struct W3Offsets {
  int pl, sc, zp;
};
struct MixedDma {
  const uint8_t* a0;  // this lane's source for group 0 of the W1 block
  int step;           // bytes per group
  int off3;           // W3 block minus W1 block
};

template <int MB, int BMIN, typename Ctx>
__device__ inline MixedDma mixed_dma(const Ctx& c, const W3Offsets& o3) {
  using SL = StageLayout<MB, BMIN>;
  constexpr int i = SL::ops - 1;
  const int slot = 64 * i + c.lane;
  MixedDma m;
  if (slot < 16 * MB) {
    m.a0 = c.pl + 16 * slot; m.step = c.pl_step; m.off3 = o3.pl;
  } else if (slot < 16 * MB + 2 * SL::levels) {
    m.a0 = c.sc + 16 * (slot - 16 * MB); m.step = c.sc_step; m.off3 = o3.sc;
  } else {
    m.a0 = c.zp; m.step = 16; m.off3 = o3.zp;
  }
  return m;
}

template <int MB, int BMIN, bool W3, typename Ctx>
__device__ inline void dma_stage(const Ctx& c, const MixedDma& m, int pl3, int g, uint8_t* st) {
  using SL = StageLayout<MB, BMIN>;
  const uint8_t* pl = c.pl + (size_t)g * c.pl_step + (W3 ? pl3 : 0);
#pragma unroll
  for (int i = 0; i < SL::ops; ++i) {
    if (64 * (i + 1) <= 16 * MB) {  // constant once the loop is unrolled
      __builtin_amdgcn_global_load_lds(D2MOE_GPTR(pl + 1024 * i + 16 * c.lane),
                                       D2MOE_LPTR(st + 1024 * i), 16, 0, kCpolNT);
    } else if (64 * i + c.lane < SL::slots) {
      const uint8_t* src = m.a0 + (size_t)g * m.step + (W3 ? m.off3 : 0);
      __builtin_amdgcn_global_load_lds(D2MOE_GPTR(src), D2MOE_LPTR(st + 1024 * i), 16, 0, 0);
    }
  }
}

// The W1 and W3 sums are independent chains, so without an ordering point
// the compiler defers a stage's scale FMAs past the next stage's LDS reads and
// keeps all of its MFMA results live (register spills).  A volatile asm that
// takes the sums after each stage ends that stage's FMAs before the next
// stage's (volatile) LDS reads.
template <int NCB>
__device__ inline void settle(v4f (&acc)[NCB]) {
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) asm volatile("" : "+v"(acc[cb]));
}

template <int MB, int BMIN, int NL, int NCB>
__device__ inline void decode_pairs(const WaveCtx<NCB>& c, const W3Offsets& o3, uint8_t* ring,
                                    int g0, int g1, v4f (&acc)[2][NCB]) {
  static_assert(kDepth == 4, "the unrolled step below assumes four stages");
  using SL = StageLayout<MB, BMIN>;
  constexpr int ND = SL::ops, NB = 2 * NL;
  constexpr int kStage = stage_bytes<BMIN>();
  const MixedDma mx = mixed_dma<MB, BMIN>(c, o3);
  const int N = 2 * (g1 - g0);  // stages
  BData<NCB> B[2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) B[i].lo[cb] = B[i].hi[cb] = v4i{0, 0, 0, 0};
  if (N <= 0) return;
  dma_stage<MB, BMIN, false>(c, mx, o3.pl, g0, ring);
  load_b<NL>(B[0], c, g0);
  if (1 < N) dma_stage<MB, BMIN, true>(c, mx, o3.pl, g0, ring + kStage);
  if (2 < N) dma_stage<MB, BMIN, false>(c, mx, o3.pl, g0 + 1, ring + 2 * kStage);
#define D2MOE_PSTEP(K)                                                                   \
  if (s + (K) < N) {                                                                     \
    const int ss = s + (K);                                                              \
    if (((K) & 1) == 0 && ss + 2 < N) load_b<NL>(B[(((K) >> 1) + 1) & 1], c, g0 + (ss >> 1) + 1); \
    if (ss + 3 < N) {                                                                    \
      dma_stage<MB, BMIN, ((K) + 3) & 1>(c, mx, o3.pl, g0 + ((ss + 3) >> 1),            \
                                         ring + (((K) + 3) % kDepth) * kStage);          \
      wait_vm<3 * ND + NB>();                                                            \
    } else if (ss + 2 < N) {                                                             \
      wait_vm<2 * ND + NB>();                                                            \
    } else if (ss + 1 < N) {                                                             \
      wait_vm<ND>();                                                                     \
    } else {                                                                             \
      wait_vm<0>();                                                                      \
    }                                                                                    \
    if (((K) & 1) == 0) ready_b(B[(K) >> 1]);                                            \
    compute_group<MB, BMIN, ((K) % kDepth) * kStage, NL>(B[(K) >> 1], c, acc[(K) & 1]); \
    settle(acc[(K) & 1]);                                                                \
  }
  for (int s = 0; s < N; s += kDepth) {
    D2MOE_PSTEP(0)
    D2MOE_PSTEP(1)
    D2MOE_PSTEP(2)
    D2MOE_PSTEP(3)
  }
#undef D2MOE_PSTEP
  // every real exit has already waited for all (its last stage waits with
  // vmcnt 0); the wait here puts one on every exit edge of the loop as well
  wait_vm<0>();
}

// elist, Xq, Xs, npos as for decode_kernel.  Each wave streams two 16-row
// blocks in alternate ring stages over 1/KS of the groups (KS waves share
// them):
//   SWIGLU: f = d_ff; the W1 block rb and the W3 block rb + f/16 of the stacked
//   W13 (rows f.. are W3), combined as silu(a) * c into h rows rb*16..;
//   otherwise (W2): f = the matrix's rows; the adjacent blocks 2p and 2p + 1,
//   written to output rows 32p.. (f / 16 must be even).
// Workgroup x covers NW / KS such units.  With KS > 1 the waves' partial sums
// meet in their (then idle) rings and the first wave of each unit finishes.
template <int NW, int KS, int NCB, int BMIN, bool SWIGLU>
__global__ __launch_bounds__(64 * NW)
__attribute__((amdgpu_waves_per_eu(NCB == 1 ? 4 : NCB == 2 ? 3 : 2)))
void decode13_kernel(MwqView W, const int32_t* __restrict__ elist, const uint8_t* __restrict__ Xq,
                     const uint32_t* __restrict__ Xs, int npos, int f, float* __restrict__ out,
                     int out_ld, uint32_t* __restrict__ rowmax) {
  constexpr int kStage = stage_bytes<BMIN>();
  static_assert(NW % KS == 0, "whole row blocks per workgroup");
  static_assert(kDepth * kStage >= 2 * NCB * 64 * 4 * (int)sizeof(float), "partial sums fit the ring");
  __shared__ __attribute__((aligned(16))) uint8_t ring[NW][kDepth * kStage];
  const int ei = blockIdx.y;
  const int e = elist[4 * ei], p0 = elist[4 * ei + 1], p1 = elist[4 * ei + 2];
  const int mb_req = elist[4 * ei + 3];
  if (mb_req == 0) return;  // workgroup-uniform
  const int mb = mb_req < W.b_max ? mb_req : W.b_max;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nrb = f / 16;
  const int unit = blockIdx.x * (NW / KS) + wave / KS;
  const int rb = SWIGLU ? unit : 2 * unit;  // first row block of the pair
  const int kp = wave % KS;
  // a row block past the end (f / 16 not a multiple of NW / KS) does no work
  // but still meets the workgroup barrier below
  const bool active = rb < nrb;
  if (KS == 1 && !active) return;
  const int NG = W.cols / G;
  const int g0 = kp * NG / KS, g1 = (kp + 1) * NG / KS;
  const int ncol = p1 - p0;

  WaveCtx<NCB> c;
  c.lane = lane;
  c.q = lane >> 4;
  c.j = lane & 15;
  const int piece = lane & 1;
  const int t = c.j >> 1;
  c.info_shift = 8 + 8 * piece;
  bool valid[NCB];
  int pos[NCB];
  {
    uint32_t iw[NCB * kDecodeCols];
#pragma unroll
    for (int i = 0; i < NCB * kDecodeCols; ++i) iw[i] = Xs[p0 + i];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const int tc = kDecodeCols * cb + t;
      valid[cb] = tc < ncol;
      pos[cb] = p0 + tc;
      const int src = valid[cb] ? pos[cb] : npos;
      const size_t base = ((size_t)src * NG) * 2 + piece;
      c.xq[cb] = Xq + base * 128 + c.q * 32 + (size_t)g0 * 256;
      c.lmask[cb] = __ballot(valid[cb]) | 1ull;
      uint32_t info = 0u;
#pragma unroll
      for (int i = 0; i < kDecodeCols; ++i) info = t == i ? iw[kDecodeCols * cb + i] : info;
      c.info[cb] = valid[cb] ? info : 0u;
    }
  }

  // the bases point at group g0, so that the stream below always starts at
  // group 0 (the same loop as an unsplit wave, with no per-wave offsets live)
  const size_t blk1 = W.block(e, rb, g0), blk3 = W.block(e, SWIGLU ? rb + nrb : rb + 1, g0);
  c.pl = (const uint8_t*)(W.planes + W.plane_word(blk1, 0, 0));
  c.sc = (const uint8_t*)(W.scales + W.scale_idx(blk1, 0, 0));
  c.zp = W.zeros + W.zero_idx(blk1, 0);
  c.pl_step = W.b_max * 64 * 4;
  c.sc_step = W.levels() * 16 * 2;
  const int dblk = (int)(blk3 - blk1);  // the launcher checks that the offsets fit
  const W3Offsets o3{dblk * c.pl_step, dblk * c.sc_step, dblk * 16};
  c.k = sigma_consts();
  {
    const uint32_t base = lds_addr(ring[wave]);
    c.lds_pl = base + 4 * lane;
    c.lds_sc = base + 8 * c.q;
    c.lds_z = base + c.j;
    c.lds_zq = base + 4 * c.q;
  }

  v4f acc[2][NCB];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[h][cb] = v4f{0.f, 0.f, 0.f, 0.f};
  if (active) {
    // as in decode_kernel: items that leave the last column block empty
    // run the group loop of one block fewer
    const bool full = ncol > kDecodeCols * (NCB - 1);
    switch (mb) {
#define D2MOE_CASE(MB)                                                                   \
  case MB:                                                                               \
    if constexpr (MB >= BMIN) {                                                          \
      if (full || NCB == 1)                                                              \
        decode_pairs<MB, BMIN, NCB>(c, o3, ring[wave], 0, g1 - g0, acc);                 \
      else                                                                               \
        decode_pairs<MB, BMIN, NCB == 1 ? 1 : NCB - 1>(c, o3, ring[wave], 0, g1 - g0, acc); \
    }                                                                                    \
    break;
      D2MOE_CASE(1) D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6)
      D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
      default: break;
    }
  }
  if constexpr (KS > 1) {
    // every DMA of this wave has completed (its last step waits for all), so
    // its ring can hold its partial sums
    float4* red = (float4*)ring[wave];
    if (kp != 0) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          red[64 * (NCB * h + cb) + lane] = float4{acc[h][cb][0], acc[h][cb][1], acc[h][cb][2], acc[h][cb][3]};
    }
    __syncthreads();
    if (kp != 0 || !active) return;
    for (int w = 1; w < KS; ++w) {
      const float4* part = (const float4*)ring[wave + w];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const float4 v = part[64 * (NCB * h + cb) + lane];
          acc[h][cb][0] += v.x; acc[h][cb][1] += v.y; acc[h][cb][2] += v.z; acc[h][cb][3] += v.w;
        }
    }
  }

  if constexpr (!SWIGLU) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float o[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = acc[h][cb][r] + __shfl_xor(acc[h][cb][r], 1, 64);
        if (valid[cb] && piece == 0)
          *(float4*)(out + (size_t)pos[cb] * out_ld + (rb + h) * 16 + 4 * c.q) =
              float4{o[0], o[1], o[2], o[3]};
      }
    return;
  }
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    float o[4];
    float m = 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float a = acc[0][cb][r] + __shfl_xor(acc[0][cb][r], 1, 64);  // hi + lo pieces
      const float u = acc[1][cb][r] + __shfl_xor(acc[1][cb][r], 1, 64);
      o[r] = silu(a) * u;
      m = fmaxf(m, fabsf(o[r]));
    }
    if (valid[cb] && piece == 0)
      *(float4*)(out + (size_t)pos[cb] * out_ld + rb * 16 + 4 * c.q) = float4{o[0], o[1], o[2], o[3]};
    if (rowmax) {
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      if (valid[cb] && piece == 0 && c.q == 0) rowmax[(size_t)pos[cb] * nrb + rb] = __float_as_uint(m);
    }
  }
}

template <typename TIN>
hipError_t run_xprep(const TIN* in, int in_ld, const int32_t* perm, int kdiv, int npos, int K,
                     const uint32_t* rowmax, int rowmax_parts, uint8_t* Xq, uint32_t* Xs,
                     const d2moe_routing* r, bool work_list, int E, int L, int32_t* elist,
                     int nitems, int item, hipStream_t s) {
  xprep_kernel<TIN><<<dim3(npos + 1, (K + kPrepCols - 1) / kPrepCols), kPrepThreads, 0, s>>>(
      in, in_ld, perm, kdiv, npos, K, rowmax, rowmax_parts, Xq, Xs, r->perm, r->topk_bits,
      work_list ? r->offsets : nullptr, work_list ? r->expert_maxbit : nullptr, E, L, elist,
      nitems, item);
  return hipGetLastError();
}

}  // namespace

// decode13_kernel addresses the second block of a wave (the W3 block of the
// same rows, or the next W2 row block) as a 32-bit byte offset from the
// first.  Layers whose offsets do not fit (W1 half of one expert's planes
// of 2 GB or more, far beyond the paper's models) take the grouped-GEMM path.
bool decode_path_ok(const d2moe_mwq* w13, const d2moe_mwq* w2, int T) {
  if (T > kDecodeMaxTokens || w13->group != 128 || w2->group != 128) return false;
  const size_t w3_off = (size_t)(w13->rows / 2 / 16) * (w13->cols / G) * (size_t)w13->b_max * 256;
  const size_t w2_off = (size_t)(w2->cols / G) * (size_t)w2->b_max * 256;
  return w3_off < ((size_t)1 << 31) && w2_off < ((size_t)1 << 31);
}

// Waves per workgroup: one per SIMD, so that the per-SIMD register budget,
// not the workgroup size, sets how many workgroups share a compute unit.
constexpr int kDecodeWaves = 4;

// The expert kernels take optional start / stop events.  Given events, the
// kernel is launched through hipExtLaunchKernel, which records them as the
// kernel's own start and end time stamps; events recorded as separate stream
// markers around the launch would also count the kernel's wait for the
// previous one (about 5 us).
template <typename K, typename... A>
inline void launch_timed(K kernel, dim3 grid, dim3 block, hipStream_t s, hipEvent_t ev0,
                         hipEvent_t ev1, A... args) {
  if (ev0 || ev1)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev0, ev1, 0, args...);
  else
    kernel<<<grid, block, 0, s>>>(args...);
}

template <int NCB>
hipError_t launch_decode_kernel(int b_min, dim3 grid, const MwqView& W, const int32_t* elist,
                                const uint8_t* Xq, const uint32_t* Xs, int npos, float* out,
                                int out_ld, hipStream_t s, hipEvent_t ev0 = nullptr,
                                hipEvent_t ev1 = nullptr) {
  switch (b_min) {
#define D2MOE_CASE(B)                                                                      \
  case B:                                                                                  \
    launch_timed(decode_kernel<kDecodeWaves, NCB, B>, grid, dim3(64 * kDecodeWaves), s,    \
                 ev0, ev1, W, elist, Xq, Xs, npos, out, out_ld);                          \
    break;
    D2MOE_CASE(1) D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6)
    D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// W1/W3 with one wave per row block (decode13_kernel), kDecodeWaves row blocks
// per workgroup.
template <int KS, int NCB, bool SWIGLU = true>
hipError_t launch_decode13_kernel(int b_min, int ny, const MwqView& W, const int32_t* elist,
                                  const uint8_t* Xq, const uint32_t* Xs, int npos, int f,
                                  float* out, int out_ld, uint32_t* rowmax, hipStream_t s,
                                  hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr) {
  constexpr int upw = kDecodeWaves / KS;        // units (row blocks or pairs) per workgroup
  const int units = SWIGLU ? f / 16 : f / 32;
  const dim3 grid((units + upw - 1) / upw, ny);
  switch (b_min) {
#define D2MOE_CASE(B)                                                                      \
  case B:                                                                                  \
    launch_timed(decode13_kernel<kDecodeWaves, KS, NCB, B, SWIGLU>, grid,                \
                 dim3(64 * kDecodeWaves), s, ev0, ev1, W, elist, Xq, Xs, npos, f, out,    \
                 out_ld, rowmax);                                                          \
    break;
    D2MOE_CASE(1) D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6)
    D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_ffn(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                             const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                             const DecodeBuffers& b, hipStream_t s, const hipEvent_t* events) {
  hipError_t err;
  const int L = w13->b_max - w13->b_min + 1;
  const int npos = T * k;
  // two column blocks per work item once experts hold more than 4 positions
  // on average (an expert's planes are then streamed once for up to 16 of
  // its positions instead of once per 8, and an item of 8 or fewer runs the
  // one-block loop of the two-block kernel, its empty block skipped): at the
  // Mixtral shape 20, 24 and 28 tokens took 0.243-0.246, 0.277 and
  // 0.290-0.295 ms per step against 0.251, 0.287 and 0.331 ms with the
  // threshold at 7.  Three above 12 on average: at 16 (64 tokens, top-2 of
  // 8) about 4 experts in 10 hold more than 16 positions, and streaming them
  // once for up to 24 took the step from 0.54-0.56 to 0.51-0.52 ms; from 7
  // or 9 instead of 12 it was slower from 32 or 40 tokens on.
  const int ncb = npos > 12 * E ? 3 : npos > 4 * E ? 2 : 1;
  const int item = ncb * kDecodeCols;
  // work items: each active expert's positions in runs of `item`
  const int ny = (E < npos ? E : npos) + (npos + item - 1) / item;
  if (xd == D2MOE_BF16)
    err = run_xprep<uint16_t>((const uint16_t*)x, d, r->perm, k, npos, d, nullptr, 0, b.xq13,
                              b.xs13, r, true, E, L, b.elist, ny, item, s);
  else
    err = run_xprep<float>((const float*)x, d, r->perm, k, npos, d, nullptr, 0, b.xq13, b.xs13,
                           r, true, E, L, b.elist, ny, item, s);
  if (err != hipSuccess) return err;
  const MwqView W13 = view_of(w13), W2 = view_of(w2);
  // the expert kernels record the caller's events themselves (launch_timed)
  const hipEvent_t e0 = events ? events[0] : nullptr, e1 = events ? events[1] : nullptr;
  const hipEvent_t e2 = events ? events[2] : nullptr, e3 = events ? events[3] : nullptr;
  const dim3 g2(d / 16, ny);
  // W1/W3: each wave streams both matrices' blocks of its rows (one
  // activation load serves both), two waves per row block, each over half of
  // the reduction, or four waves over a quarter each when the two-wave grid
  // would not fill the GPU's 4096 wave slots (one or two active experts:
  // the dense FFN, batch 1), so that more streams are in flight.
  // decode_path_ok has checked that the W3 block's 32-bit offset fits.
  const long active_items = E < npos ? E : npos;
  const bool ks4 = (long)(d_ff / 16) * active_items * 2 < 4096;
  if (ncb == 1)
    err = ks4 ? launch_decode13_kernel<4, 1>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1)
              : launch_decode13_kernel<2, 1>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1);
  else if (ncb == 2)
    err = ks4 ? launch_decode13_kernel<4, 2>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1)
              : launch_decode13_kernel<2, 2>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1);
  else
    err = ks4 ? launch_decode13_kernel<4, 3>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1)
              : launch_decode13_kernel<2, 3>(w13->b_min, ny, W13, b.elist, b.xq13, b.xs13, npos,
                                             d_ff, b.h32, d_ff, b.hmax, s, e0, e1);
  if (err != hipSuccess) return err;
  err = run_xprep<float>(b.h32, d_ff, nullptr, 1, npos, d_ff, b.hmax, d_ff / 16, b.xq2, b.xs2, r,
                         false, E, L, nullptr, 0, item, s);
  if (err != hipSuccess) return err;
  // W2: when the grid still fills the GPU's wave slots
  // (256 CUs x 16 waves) about 1.25 times over, each wave streams a pair of
  // adjacent row blocks over a quarter of the reduction (decode13_kernel, one
  // activation load for both blocks); with fewer work items (batches below
  // 8 at the Mixtral shape) the 4-wave-per-row-block kernel keeps more
  // streams in flight and is faster.  The second block's offset is one row
  // block of groups.
  constexpr int kW2Split = 4;
  const bool pairs2 = (d / 16) % 2 == 0 && (long)(d / 32) * ny * kW2Split >= 5120;
  if (pairs2 && ncb == 1)
    err = launch_decode13_kernel<kW2Split, 1, false>(w2->b_min, ny, W2, b.elist, b.xq2, b.xs2,
                                                     npos, d, b.y, d, nullptr, s, e2, e3);
  else if (pairs2 && ncb == 2)
    err = launch_decode13_kernel<kW2Split, 2, false>(w2->b_min, ny, W2, b.elist, b.xq2, b.xs2,
                                                     npos, d, b.y, d, nullptr, s, e2, e3);
  else if (pairs2)
    err = launch_decode13_kernel<kW2Split, 3, false>(w2->b_min, ny, W2, b.elist, b.xq2, b.xs2,
                                                     npos, d, b.y, d, nullptr, s, e2, e3);
  else
    err = ncb == 1   ? launch_decode_kernel<1>(w2->b_min, g2, W2, b.elist, b.xq2, b.xs2, npos,
                                               b.y, d, s, e2, e3)
          : ncb == 2 ? launch_decode_kernel<2>(w2->b_min, g2, W2, b.elist, b.xq2, b.xs2, npos,
                                               b.y, d, s, e2, e3)
                     : launch_decode_kernel<3>(w2->b_min, g2, W2, b.elist, b.xq2, b.xs2, npos,
                                               b.y, d, s, e2, e3);
  if (err != hipSuccess) return err;
  return hipSuccess;
}

}  // namespace d2moe
