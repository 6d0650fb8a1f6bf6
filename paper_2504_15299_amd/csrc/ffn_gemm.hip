// Grouped mixed-bit expert GEMM (Sec. 3.3.2: dequantization fused with the
// expert matrix products) for any number of tokens per expert, and the
// weighted combine (Fig. 1: outputs of the activated experts weighted by the
// gate).
//
// Positions are the (token, slot) pairs sorted by (expert, bit-width), so an
// (expert, bit-width) bucket is a contiguous run of positions that all read
// the same b-bit prefix of the expert's planes.  Buckets are cut into chunks
// of at most kChunk = 256 positions; one 4-wave workgroup computes one chunk
// against 128 weight rows, and two such workgroups share a compute unit.
// Each wave owns 64 positions, and all share one dequantized weight tile, so
// a weight is dequantized once per chunk however many positions it holds.
// Chunks of at most 64 positions can run in an 8-wave variant in which every
// wave takes 16 of the tile's rows for the same positions.
//
// Per reduction step of 32 columns (one plane word per row):
//   * the LDS DMA engine brings the raw planes, scales and zero points of a
//     later step into a ring shared by the workgroup, and each wave's
//     gathered activation rows of a later step into its own ring;
//   * the workgroup dequantizes the next step's 128 x 32 tile into bf16 while
//     each wave runs the current step's v_mfma_f32_16x16x32_bf16 products
//     (its positions x 128 rows, fp32 accumulation) from the other tile
//     buffer, the products interleaved with the dequantization's vector
//     instructions;
//   * one barrier per step orders the shared buffers.
// The W1/W3 variant puts 64 rows of W1 and the same 64 rows of W3 in one tile,
// so a lane holds a and c of the same output and applies SwiGLU in registers.
#include <type_traits>

#include "internal.h"

namespace d2moe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaveM = 64;                  // positions per wave
// waves per workgroup: 4 in the wide kernel (one per SIMD, two workgroups
// per compute unit), 8 in the narrow one
template <bool NARROW> constexpr int n_waves() { return NARROW ? 8 : 4; }
constexpr int kChunk = n_waves<false>() * kWaveM;  // positions per chunk
constexpr int kTileRows = 128;              // weight rows per workgroup
constexpr int kStepK = 32;                  // reduction columns per step
// activation lookahead in steps: one in the wide kernel (its 2-stage ring
// leaves LDS for the tiles; the activations mostly come from L2), two in the
// narrow one
template <bool NARROW> constexpr int x_lead() { return NARROW ? 2 : 1; }
constexpr int kXStage = kWaveM * kStepK * 2;  // bytes per wave and stage
// Raw stage layout at MB planes and LS scale levels (bytes): plane p at
// 512 p (one word per tile row), the scales of level l at 512 MB + 256 l (one
// binary16 per tile row), then the zero points (one byte per tile row).
// 16-byte DMA slots 0 .. raw_slots - 1 carry them; DMA instruction i of wave
// w moves slots 256 i + 64 w .. + 63 (one instruction per wave in the 8-wave
// kernel, two in the 4-wave one).  The ring holds as many stages as fit
// kRawBytes, at most 8 (4 at 7 and 8 bits, 8 at 2 to 4), so the DMA runs
// further ahead of the dequantization when a step has less to read.
constexpr int kRawBytes = 25088;
constexpr int raw_zero_off(int MB, int LS) { return 512 * MB + 256 * LS; }
constexpr int raw_stage_bytes(int MB, int LS) { return raw_zero_off(MB, LS) + 128; }
constexpr int raw_slots(int MB, int LS) { return raw_stage_bytes(MB, LS) / 16; }
constexpr int raw_ring(int MB, int LS) {
  return kRawBytes / raw_stage_bytes(MB, LS) < 8 ? kRawBytes / raw_stage_bytes(MB, LS) : 8;
}
static_assert(raw_ring(8, 8) >= 4, "at least 4 raw stages");
template <bool NARROW> constexpr int raw_dmas() { return NARROW ? 1 : 2; }
constexpr int kWTile = kTileRows * kStepK * 2;  // dequantized bf16 tile bytes

#define D2MOE_GPTR(p) ((__attribute__((address_space(1))) void*)(p))
#define D2MOE_LPTR(p) ((__attribute__((address_space(3))) void*)(p))

// Chunk table, written on the device from the routing histogram:
// chunks[4 c] = first position, positions (0: no work), bit-width, expert.
// Buckets are taken in order of bit-width (widest first: a workgroup's time
// grows with the planes it dequantizes), then of size (largest first, ties
// in bucket order), so that the longest workgroups start first.  One
// workgroup of kChunkThreads threads, one bucket per thread (nb <=
// kChunkThreads, bucket index < 1024).
constexpr int kChunkThreads = 512;
__global__ __launch_bounds__(kChunkThreads) void chunk_kernel(
    const int32_t* __restrict__ hist, const int32_t* __restrict__ offsets, int nb, int L, int b_min,
    int one_cnt, int one_bit, int one_cs, int n_ub, int32_t* __restrict__ chunks) {
  __shared__ unsigned long long key[kChunkThreads];
  __shared__ int scan[kChunkThreads];
  const int j = threadIdx.x;
  if (hist == nullptr) {  // one bucket: every position, expert 0, chunks of one_cs
    for (int c = j; c < n_ub; c += kChunkThreads) {
      const int m0 = c * one_cs;
      chunks[4 * c] = m0;
      chunks[4 * c + 1] = m0 < one_cnt ? min(one_cs, one_cnt - m0) : 0;
      chunks[4 * c + 2] = one_bit;
      chunks[4 * c + 3] = 0;
    }
    return;
  }
  // sort buckets by (bit-width, size) descending, index ascending: bitonic
  // sort of one 64-bit key per thread, the width level in bits 50..53, size
  // in bits 10..49 and 1023 - index in the low ten (empty buckets have key 0
  // and sort last)
  const int cj = j < nb ? hist[j] : 0;
  key[j] = j < nb && cj > 0 ? ((unsigned long long)(j % L + 1) << 50) |
                                  ((unsigned long long)cj << 10) | (unsigned)(1023 - j)
                            : 0ull;
  __syncthreads();
  for (int kk = 2; kk <= kChunkThreads; kk <<= 1) {
    for (int jj = kk >> 1; jj > 0; jj >>= 1) {
      const int ix = j ^ jj;
      if (ix > j) {
        const unsigned long long a = key[j], b = key[ix];
        const bool desc = (j & kk) == 0;  // this pair's segment runs descending
        if (desc ? a < b : a > b) {
          key[j] = b;
          key[ix] = a;
        }
      }
      __syncthreads();
    }
  }
  // chunks of the bucket at sorted position j, and their exclusive prefix
  const unsigned long long kj = key[j];
  const int cnt_j = (int)((kj >> 10) & ((1ull << 40) - 1)), bkt = 1023 - (int)(kj & 1023ull);
  const int nch_j = (cnt_j + kChunk - 1) / kChunk;
  scan[j] = nch_j;
  __syncthreads();
  for (int off = 1; off < kChunkThreads; off <<= 1) {
    const int v = j >= off ? scan[j - off] : 0;
    __syncthreads();
    scan[j] += v;
    __syncthreads();
  }
  const int first = scan[j] - nch_j;
  const int total = scan[kChunkThreads - 1];
  if (nch_j > 0) {
    const int b0 = offsets[bkt];
    for (int q = 0; q < nch_j; ++q) {
      const int c = first + q;
      if (c >= n_ub) break;
      chunks[4 * c] = b0 + q * kChunk;
      chunks[4 * c + 1] = min(kChunk, cnt_j - q * kChunk);
      chunks[4 * c + 2] = b_min + bkt % L;
      chunks[4 * c + 3] = bkt / L;
    }
  }
  for (int c = total + j; c < n_ub; c += kChunkThreads) chunks[4 * c + 1] = 0;
}

__device__ inline float silu(float a) { return a / (1.0f + __expf(-a)); }

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 b2 __attribute__((ext_vector_type(2)));

__device__ inline h2 as_h2(uint32_t v) { return __builtin_bit_cast(h2, v); }
__device__ inline uint32_t as_u(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ inline uint32_t h2_splat(float v) {
  const _Float16 h = (_Float16)v;
  return as_u(h2{h, h});
}

// LDS accesses to the DMA-filled rings and to the shared tile are inline
// assembly: with LDS DMA in flight the compiler would otherwise wait for every
// outstanding vector-memory instruction (draining the prefetch) before each
// LDS access it cannot prove independent.  Reads are ordered by an explicit
// lgkmcnt wait and re-bound after it.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// OFF is the instruction's unsigned 16-bit byte offset added to the address.
template <int OFF = 0>
__device__ inline void ld128(u32x4& v, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF) : "memory");
}
template <int OFF = 0>
__device__ inline void ld32(uint32_t& v, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF) : "memory");
}
template <int OFF = 0>
__device__ inline void ldu16(uint32_t& v, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  asm volatile("ds_read_u16 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF) : "memory");
}
template <int OFF = 0>
__device__ inline void ldu8(uint32_t& v, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  asm volatile("ds_read_u8 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF) : "memory");
}
__device__ inline void st64(uint32_t a, uint32_t lo, uint32_t hi) {
  asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"(u32x2{lo, hi}) : "memory");
}
__device__ inline void st128(uint32_t a, uint32_t x, uint32_t y, uint32_t z, uint32_t w) {
  asm volatile("ds_write_b128 %0, %1" ::"v"(a), "v"(u32x4{x, y, z, w}) : "memory");
}
__device__ inline void wait_lgkm() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ inline void bar() { __builtin_amdgcn_s_barrier(); }

// 16-byte chunk q of tile row r sits at chunk q ^ ((r >> 2) & 3), so that the
// 16 rows one MFMA operand read touches fall in distinct banks.
__device__ inline uint32_t swz(int r, int q) { return (uint32_t)(r * 64 + ((q ^ ((r >> 2) & 3)) << 4)); }

// f(integral_constant<int, i>) for i = 0 .. N-1, so that the index can be a
// template argument (an instruction offset) inside f.
template <int N, int I = 0, typename F>
__device__ __attribute__((always_inline)) inline void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// Registers of one step: raw words, scales and zero point of the tile row a
// thread dequantizes, and the MFMA operands of its wave.
struct StepRegs {
  uint32_t w[8];   // plane words
  uint32_t sp[8];  // binary16 scale of plane p (p >= b_min); register index = plane
  uint32_t s1, z;  // base scale and zero point
  u32x4 A[4], B[4], B2[4];  // B, B2: weight operands of tile rows 0..63, 64..127
  // Re-binds, after the covering wait, the registers the inline-asm LDS reads
  // of a step wrote: MB plane words, the scales of planes SPLO..MB-1, and
  // the operands of NA A, NB B and NB2 B2 reads.
  template <int MB, int SPLO, int NA, int NB, int NB2>
  __device__ __attribute__((always_inline)) inline void rebind() {
#pragma unroll
    for (int p = 0; p < MB; ++p) asm volatile("" : "+v"(w[p]));
#pragma unroll
    for (int p = SPLO; p < MB; ++p) asm volatile("" : "+v"(sp[p]));
    asm volatile("" : "+v"(s1));
    asm volatile("" : "+v"(z));
#pragma unroll
    for (int i = 0; i < NA; ++i) asm volatile("" : "+v"(A[i]));
#pragma unroll
    for (int i = 0; i < NB; ++i) asm volatile("" : "+v"(B[i]));
#pragma unroll
    for (int i = 0; i < NB2; ++i) asm volatile("" : "+v"(B2[i]));
  }
};

// Dequantization of four weight pairs (columns j, j + 16 for
// j = 4 dq .. 4 dq + 3) of a tile row at MB planes into bf16 pairs for the
// tile (o[0..1] columns 4 dq .. 4 dq + 3, o[2..3] columns 16 + 4 dq ..).
// It works on pairs in packed fp16: shifting a plane word left by 15 - j puts
// bit j at bit 15 and bit j + 16 at bit 31, the sign positions of the two
// halves, and one and-or turns the pair into (+-c_p, +-c_p).  With every plane
// read as a sign,
//   W^_b = s1 (Q - z) + sum_{p>=b_min} s_p sigma_p
//        = C + sum_{p<b} c_p (2 bit_p - 1),  c_p = s1 2^(p-1) for p < b_min,
//          c_p = s_p for p >= b_min,  C = s1 ((2^b_min - 1) / 2 - z),
// accumulated in fp16 from C, then rounded to bf16 for the MFMA.  Every scale
// is >= 0, so the sign bits of c_p are clear and the and-or only has to set
// them from the plane bits.  Rows past the matrix edge are dequantized from
// whatever their stage holds: they only reach output columns that are not
// stored.
// BMIN > 0 fixes b_min at compile time (the common ladder starts at 2 bits);
// BMIN == 0 takes it from `b_min_rt`.
template <int MB, int BMIN>
__device__ __attribute__((always_inline)) inline void dequant_pairs(
    const StepRegs& R, int b_min_rt, uint32_t sh_m, int dq, uint32_t (&o)[4]) {
  const int b_min = BMIN > 0 ? BMIN : b_min_rt;
  const float s1 = h2f((uint16_t)R.s1);
  const uint32_t C = h2_splat(s1 * ((float)((1 << b_min) - 1) * 0.5f - (float)R.z));
  // base scale as a binary16 pair; the pair of a residual plane is its scale
  // bits duplicated, and that of a base plane p < b_min is s1 2^(p-1), a
  // power-of-two multiple in binary16
  const h2 s1p = as_h2(R.s1 | (R.s1 << 16));
  h2 a[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) a[j] = as_h2(C);
#pragma unroll
  for (int p = 0; p < MB; ++p) {
    const _Float16 k = (_Float16)((float)(1 << p) * 0.5f);
    const uint32_t cp = p < b_min ? as_u(s1p * h2{k, k}) : (R.sp[p] | (R.sp[p] << 16));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t t = R.w[p] << (15 - (4 * dq + j));
      const uint32_t v = (sh_m & t) | cp;  // bit set -> -c_p
      a[j] = a[j] - as_h2(v);
    }
  }
  // (column j, column j + 16) fp16 pairs to bf16 pairs of adjacent columns
  f2 f[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) f[j] = __builtin_convertvector(a[j], f2);
  auto pk = [](float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{lo, hi}, b2));
  };
  o[0] = pk(f[0].x, f[1].x);  // columns 4 dq, 4 dq + 1
  o[1] = pk(f[2].x, f[3].x);  // 4 dq + 2, 4 dq + 3
  o[2] = pk(f[0].y, f[1].y);  // 16 + 4 dq, ...
  o[3] = pk(f[2].y, f[3].y);
}

// One workgroup: chunk blockIdx.y of the chunk table against weight-row tile
// blockIdx.x.
//   in:  bf16 activations; position p reads row (perm ? perm[p] / kdiv : p)
//   SWIGLU: W is [2f][K] (w13); the tile holds W1 rows n0..n0+63 (tile rows
//           0..63) and W3 rows f+n0.. (tile rows 64..127); out = h [pos][f] bf16
//   else:   W is [N][K], out = y [pos][N] fp32
// `expert_fixed` >= 0 overrides the chunk's expert (the shared expert).
template <int G, bool SWIGLU, bool NARROW>
__global__ __launch_bounds__(64 * n_waves<NARROW>())
__attribute__((amdgpu_waves_per_eu(NARROW ? 4 : 2))) void bgemm_kernel(
    const uint16_t* __restrict__ in, int in_ld, const int32_t* __restrict__ perm, int kdiv,
    MwqView W, const int32_t* __restrict__ chunks, int f, int N, void* __restrict__ out,
    int out_ld, int split, size_t out_split) {
  // narrow chunks stage only the chunk's shared activations (54 KB of LDS
  // in all: three workgroups per compute unit), wide ones each wave's
  // (73 KB: two)
  constexpr int NWV = n_waves<NARROW>(), RD = raw_dmas<NARROW>();
  constexpr int XL = x_lead<NARROW>(), kXRing = XL + 1;
  __shared__ __attribute__((aligned(16))) uint8_t xring[kXRing][NARROW ? 1 : NWV][kXStage];
  __shared__ __attribute__((aligned(16))) uint8_t rraw[kRawBytes];  // ring of raw stages
  __shared__ __attribute__((aligned(16))) uint8_t wtile[2][kWTile];
  __shared__ __attribute__((aligned(16))) uint8_t dummy[1][16];
  constexpr int BR = 2048 / G, SPG = G / kStepK;  // rows per block, steps per group

  const int ci = blockIdx.y;
  const int m_first = chunks[4 * ci], m_cnt = chunks[4 * ci + 1];
  const int bits = chunks[4 * ci + 2], expert = chunks[4 * ci + 3];
  if (m_cnt == 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = blockIdx.x * (SWIGLU ? kTileRows / 2 : kTileRows);
  // reduction part blockIdx.z of gridDim.z (the plain variant only): steps
  // [s_lo, s_lo + nsteps), partial sums to plane blockIdx.z of `out`
  const int K = W.cols, b_min = W.b_min;
  const int s_all = K / kStepK;
  const int s_lo = SWIGLU ? 0 : (int)((long)blockIdx.z * s_all / gridDim.z);
  const int nsteps = SWIGLU ? s_all : (int)((long)(blockIdx.z + 1) * s_all / gridDim.z) - s_lo;
  if (!SWIGLU) out = (float*)out + (size_t)blockIdx.z * out_split;
  const int nlev = bits - b_min + 1;
  const int nout = SWIGLU ? f : N;
  const bool active = kWaveM * wave < m_cnt;  // wave-uniform
  // Narrow chunk (at most one wave's 64 positions): instead of one wave
  // running all 32 products of a step while seven wait at the barrier, every
  // wave takes a share of the tile's rows for those positions (W2: 16 rows
  // each; W1/W3: one 16-row block of W1 and the same block of W3, for 32 of
  // the 64 positions), reading the activations that wave 0 stages.  When
  // `split` is set, narrow and wide chunks run in two launches of the two
  // instantiations of this kernel (one MFMA path each keeps the register
  // allocation of either unchanged), each skipping the other's chunks;
  // otherwise the wide one takes every chunk.
  constexpr bool narrow = NARROW;
  if (NARROW ? m_cnt > kWaveM : (split && m_cnt <= kWaveM)) return;

  // ---- raw weight DMA: 16-byte slot u of a stage laid out for MB planes
  // and LS scale levels ----
  // global row of tile row r
  auto grow = [&](int r) { return SWIGLU ? (r < 64 ? n0 + r : f + n0 + r - 64) : n0 + r; };
  auto row_ok = [&](int r) { return SWIGLU ? n0 + (r & 63) < f : n0 + r < N; };
  struct RawSlot {
    const uint8_t* src;  // address at step 0
    int sb, sc;          // bytes per group, per 32-column step
    bool real;
  };
  auto raw_slot = [&](int u, int MB, int LS) {
    RawSlot q{(const uint8_t*)W.planes, 0, 0, false};
    const int u1 = 32 * MB, u2 = u1 + 16 * LS;
    if (u < u1) {  // plane p = u / 32, tile rows 4 v .. 4 v + 3 of it
      const int p = u >> 5, v = u & 31;
      const int r = 4 * v;  // first tile row of the slot
      if (p < bits && row_ok(r)) {
        const int gr = grow(r);
        const size_t blk = W.block(expert, gr / BR, 0);
        q = {(const uint8_t*)(W.planes + W.plane_word(blk, p, gr % BR)), W.b_max * 64 * 4, BR * 4,
             true};
      }
    } else if (u < u2) {  // level l, tile rows 8 v .. 8 v + 7
      const int l = (u - u1) >> 4, v = (u - u1) & 15;
      const int r = 8 * v;
      if (l < nlev && row_ok(r)) {
        const int gr = grow(r);
        const size_t blk = W.block(expert, gr / BR, 0);
        q = {(const uint8_t*)(W.scales + W.scale_idx(blk, l, gr % BR)), W.levels() * BR * 2, 0,
             true};
      }
    } else if (u < u2 + 8) {  // zero points, tile rows 16 z .. 16 z + 15
      const int z = u - u2;
      const int r = 16 * z;
      if (row_ok(r)) {
        const int gr = grow(r);
        const size_t blk = W.block(expert, gr / BR, 0);
        q = {W.zeros + W.zero_idx(blk, gr % BR), BR, 0, true};
      }
    }
    return q;
  };

  // ---- activation DMA: an instruction moves 16 positions' 64-byte rows.
  // Wide: wave w stages its own 64 positions, instruction i the rows
  // 16 i .. 16 i + 15 (XD = 4 per step).  Narrow: the chunk's (at most) 64
  // positions are shared, wave w < 4 stages rows 16 w .. 16 w + 15 and the
  // others issue one lane-0 load to the dummy area (XD = 1 per step), so
  // that every wave counts the same memory instructions.
  constexpr int XD = NARROW ? 1 : 4;
  const uint16_t* xsrc[XD];
#pragma unroll
  for (int i = 0; i < XD; ++i) {
    const int rl = 16 * (NARROW ? (wave & 3) : i) + (lane >> 2);
    int pos = m_first + (NARROW ? 0 : kWaveM * wave) + rl;
    pos = pos < m_first + m_cnt ? pos : m_first + m_cnt - 1;
    const int src = perm ? perm[pos] / kdiv : pos;
    const int q = (lane & 3) ^ ((rl >> 2) & 3);
    xsrc[i] = in + (size_t)src * in_ld + 8 * q;
  }
  const bool xissue = NARROW ? (wave < 4 || lane == 0) : (active || lane == 0);
  auto x_dma = [&](int step) {
    const int st = s_lo + (step < nsteps ? step : nsteps - 1);
#pragma unroll
    for (int i = 0; i < XD; ++i) {
      uint8_t* dst = NARROW ? (wave < 4 ? xring[step % kXRing][0] + 1024 * wave : dummy[0])
                            : xring[step % kXRing][wave] + 1024 * i;
      if (xissue)
        __builtin_amdgcn_global_load_lds(D2MOE_GPTR(xsrc[i] + kStepK * st), D2MOE_LPTR(dst), 16,
                                         0, 0);
    }
  };

  // ---- dequantization: tile row dr, columns 4 dq .. 4 dq + 3 and +16 for
  // dq = dq0 .. dq0 + NDQ - 1 (8 waves: one dq per thread; 4 waves: two) ----
  constexpr int NDQ = 8 / NWV;
  const int dr = tid / (4 / NDQ), dq0 = (tid % (4 / NDQ)) * NDQ;
  uint32_t sh_m;  // opaque copy of the sign mask: keeps v_bfi on registers
  asm volatile("" : "=v"(sh_m) : "0"(0x80008000u));
  const int fr = lane & 15, fq = lane >> 4;

  f32x4 acc[4][8];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The step loop is compiled for the chunk's bit-width MB (and for b_min 2,
  // the common nest start, or any b_min) and separately for waves that
  // multiply and waves that only dequantize: every LDS read of a step, its
  // products and its dequantization then form one branch-free block, in which
  // the products are interleaved with the dequantization's vector
  // instructions so that the matrix pipe and the vector ALU overlap.
  auto run = [&](auto mb_c, auto bmin_c) {
    constexpr int MB = decltype(mb_c)::value, BMIN = decltype(bmin_c)::value;
    // scale levels reserved per stage: exact when b_min is fixed, else MB
    constexpr int LS = BMIN > 0 ? MB - BMIN + 1 : MB;
    constexpr int SB = raw_stage_bytes(MB, LS), NS = raw_slots(MB, LS);
    constexpr int kRawRing = raw_ring(MB, LS);
    constexpr int SOFF = 512 * MB, ZOFF = raw_zero_off(MB, LS);

    // instruction i of this wave: slots ubase + lane, ubase = 256 i + 64 wave.
    // Every wave issues RD raw DMAs per step (lane 0 at least), so that all
    // waves count the same memory instructions: lanes whose slot is past the
    // stage issue nothing, and an instruction with no slot of its own writes
    // the dummy area from lane 0.
    RawSlot rs[RD];
    bool rissue[RD];
#pragma unroll
    for (int i = 0; i < RD; ++i) {
      rs[i] = raw_slot(256 * i + 64 * wave + lane, MB, LS);
      rissue[i] = rs[i].real || lane == 0;
    }
    auto raw_dma = [&](int step) {
      const int st = s_lo + (step < nsteps ? step : nsteps - 1);  // past the end: reload, unused
#pragma unroll
      for (int i = 0; i < RD; ++i) {
        const int ubase = 256 * i + 64 * wave;  // wave-uniform
        const uint8_t* src = rs[i].src + (size_t)(st / SPG) * rs[i].sb + (st % SPG) * rs[i].sc;
        uint8_t* dst = ubase < NS ? &rraw[(step % kRawRing) * SB + 16 * ubase] : dummy[0];
        if (rissue[i])
          __builtin_amdgcn_global_load_lds(D2MOE_GPTR(src), D2MOE_LPTR(dst), 16, 0, 0);
      }
    };

    // ---- prologue: raw 0..kRawRing-1 and activations 0..XL-1 in flight.
    // Issue order: raw 0 .. raw kRawRing-2, x 0, raw kRawRing-1 (, x 1); the
    // wait leaves the instructions after raw 0 outstanding (RD per raw stage,
    // XD per activation stage), i.e. raw 0 has landed.
#pragma unroll
    for (int i = 0; i + 1 < kRawRing; ++i) raw_dma(i);
    x_dma(0);
    raw_dma(kRawRing - 1);
    if constexpr (XL == 2) x_dma(1);
    wait_vm<(kRawRing - 1) * RD + XD + (XL == 2 ? XD : 0)>();
    bar();

    StepRegs R;
    // One step: the products of `mstep` (if MMA) from the tile buffer and
    // activation stage written in earlier steps, and the dequantization of
    // tile `dstep` from its raw stage into the other tile buffer.  `dma`
    // issues the DMA of later steps once this step's LDS reads are issued, so
    // that its issue overlaps their latency (it writes only stages that this
    // step does not read).
    auto step = [&](int dstep, int mstep, auto mma_c, auto&& dma) {
      constexpr bool MMA = decltype(mma_c)::value;
      // one address register per access width: the stage base plus this
      // thread's row, with the plane, level and operand block as offsets
      const uint32_t rb = lds_addr(rraw + (dstep % kRawRing) * SB);
      const uint32_t rb4 = rb + 4 * dr, rb2 = rb + 2 * dr, rb1 = rb + dr;
      static_for<MB>([&](auto pc) {
        constexpr int P = decltype(pc)::value;
        ld32<512 * P>(R.w[P], rb4);
      });
      ldu16<SOFF>(R.s1, rb2);
      static_for<MB>([&](auto pc) {  // level p - b_min + 1 holds the scale of plane p
        constexpr int P = decltype(pc)::value;
        if constexpr (BMIN > 0) {
          if constexpr (P >= BMIN) ldu16<SOFF + 256 * (P - BMIN + 1)>(R.sp[P], rb2);
        } else if constexpr (P >= 1) {  // below b_min the base scale is read and not used
          const int lvl = P >= b_min ? P - b_min + 1 : 0;
          ldu16(R.sp[P], rb2 + SOFF + 256 * lvl);
        }
      });
      ldu8<ZOFF>(R.z, rb1);
      // a 16-row operand block m starts 1024 m bytes after block 0 (the
      // swizzle depends on the row within the block only)
      const uint32_t wb = lds_addr(wtile[mstep & 1]) + swz(fr, fq);
      if constexpr (MMA) {
        if constexpr (NARROW) {
          const uint32_t xb = lds_addr(xring[mstep % kXRing][0]) + swz(fr, fq);
          if constexpr (SWIGLU) {
            const int mh = wave >> 2, rbw = wave & 3;
            ld128<0>(R.A[0], xb + 2048 * mh);
            ld128<1024>(R.A[1], xb + 2048 * mh);
            ld128<0>(R.B[0], wb + 1024 * rbw);
            ld128<4096>(R.B[1], wb + 1024 * rbw);
          } else {
            static_for<4>([&](auto mc) {
              constexpr int M = decltype(mc)::value;
              ld128<1024 * M>(R.A[M], xb);
            });
            ld128<0>(R.B[0], wb + 1024 * wave);
          }
        } else {
          const uint32_t xb = lds_addr(xring[mstep % kXRing][wave]) + swz(fr, fq);
          static_for<4>([&](auto mc) {
            constexpr int M = decltype(mc)::value;
            ld128<1024 * M>(R.A[M], xb);
            ld128<1024 * M>(R.B[M], wb);
            ld128<1024 * (4 + M)>(R.B2[M], wb);
          });
        }
      }
      dma();
      wait_lgkm();
      constexpr int NA = !MMA ? 0 : NARROW && SWIGLU ? 2 : 4;
      constexpr int NB = !MMA ? 0 : !NARROW ? 4 : SWIGLU ? 2 : 1;
      R.template rebind<MB, (BMIN > 0 ? BMIN : 1), NA, NB, (MMA && !NARROW ? 4 : 0)>();
      constexpr int n_mfma = !MMA ? 0 : NARROW ? 4 : 32;
      if constexpr (MMA) {
        if constexpr (NARROW) {
          if constexpr (SWIGLU) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, R.A[i]), __builtin_bit_cast(bf16x8, R.B[0]), acc[i][0],
                  0, 0, 0);
              acc[i][4] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, R.A[i]), __builtin_bit_cast(bf16x8, R.B[1]), acc[i][4],
                  0, 0, 0);
            }
          } else {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
              acc[mt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, R.A[mt]), __builtin_bit_cast(bf16x8, R.B[0]),
                  acc[mt][0], 0, 0, 0);
          }
        } else {
#pragma unroll
          for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < 8; ++nt)
              acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, R.A[mt]),
                  __builtin_bit_cast(bf16x8, nt < 4 ? R.B[nt] : R.B2[nt - 4]), acc[mt][nt], 0, 0, 0);
        }
      }
      const uint32_t wd = lds_addr(wtile[dstep & 1]);
      if constexpr (NDQ == 1) {
        uint32_t o[4];
        dequant_pairs<MB, BMIN>(R, b_min, sh_m, dq0, o);
        st64(wd + swz(dr, dq0 >> 1) + 8 * (dq0 & 1), o[0], o[1]);
        st64(wd + swz(dr, 2 + (dq0 >> 1)) + 8 * (dq0 & 1), o[2], o[3]);
      } else {  // dq0 even: the two halves of 16-byte chunks dq0 / 2 and 2 + dq0 / 2
        uint32_t o0[4], o1[4];
        dequant_pairs<MB, BMIN>(R, b_min, sh_m, dq0, o0);
        dequant_pairs<MB, BMIN>(R, b_min, sh_m, dq0 + 1, o1);
        st128(wd + swz(dr, dq0 >> 1), o0[0], o0[1], o1[0], o1[1]);
        st128(wd + swz(dr, 2 + (dq0 >> 1)), o0[2], o0[3], o1[2], o1[3]);
      }
      if constexpr (n_mfma > 0) {
        // one product, then its share of the dequantization's vector
        // instructions (about 12 per plane and 40 more per step and dq)
        constexpr int nv = (NDQ * (12 * MB + 30) + 10 + n_mfma - 1) / n_mfma;
#pragma unroll
        for (int i = 0; i < n_mfma; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, nv, 0);
        }
      }
      wait_lgkm();
    };

    // Tile 0 first; then step s issues raw s+kRawRing and activations s+XL
    // (RD and XD instructions), dequantizes s+1 and multiplies s.  With XL = 2
    // (order raw, x) the instructions issued after the activations of s, at
    // the top of step s, are the RD + XD of step s-1 (raw s+kRawRing-1,
    // activations s+1); with XL = 1 (order x, raw) the RD of raw
    // s+kRawRing-1.  Raw s+1 was issued before the activations of s
    // (kRawRing > 3), so that wait makes both this wave's raw s+1 and its
    // activations of s ready; the barrier then makes every
    // wave's raw s+1 and tile s visible, and retires all reads of the stages
    // and the tile buffer that this step overwrites.  In the last step the
    // dequantization works on a reloaded stage and its tile is never read.
    step(0, 0, std::false_type{}, [] {});
    auto loop = [&](auto mma_c) {
      for (int s = 0; s < nsteps; ++s) {
        wait_vm<XL == 2 ? RD + XD : RD>();
        bar();
        step(s + 1, s, mma_c, [&] {
          if constexpr (XL == 2) {
            raw_dma(s + kRawRing);
            x_dma(s + 2);
          } else {
            x_dma(s + 1);
            raw_dma(s + kRawRing);
          }
        });
      }
    };
    if (active || narrow)
      loop(std::true_type{});
    else
      loop(std::false_type{});
  };
  using std::integral_constant;
  if (b_min == 2) {
    switch (bits) {
#define D2MOE_CASE(MB) \
  case MB: run(integral_constant<int, MB>{}, integral_constant<int, 2>{}); break;
      D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6) D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
      default: break;
    }
  } else {
    switch (bits) {
#define D2MOE_CASE(MB) \
  case MB: run(integral_constant<int, MB>{}, integral_constant<int, 0>{}); break;
      D2MOE_CASE(1) D2MOE_CASE(2) D2MOE_CASE(3) D2MOE_CASE(4) D2MOE_CASE(5) D2MOE_CASE(6)
      D2MOE_CASE(7) D2MOE_CASE(8)
#undef D2MOE_CASE
      default: break;
    }
  }
  wait_vm<0>();  // no DMA may still be writing this workgroup's LDS at exit

  // ---- epilogue ----
  if constexpr (NARROW) {
    if constexpr (SWIGLU) {
      const int mh = wave >> 2, n = n0 + 16 * (wave & 3) + (lane & 15);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 32 * mh + 16 * i + 4 * (lane >> 4) + r;
          if (m >= m_cnt || n >= f) continue;
          ((uint16_t*)out)[(size_t)(m_first + m) * out_ld + n] =
              f2bf(silu(acc[i][0][r]) * acc[i][4][r]);
        }
    } else {
      const int n = n0 + 16 * wave + (lane & 15);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * mt + 4 * (lane >> 4) + r;
          if (m >= m_cnt || n >= N) continue;
          ((float*)out)[(size_t)(m_first + m) * out_ld + n] = acc[mt][0][r];
        }
    }
    return;
  }
  if (!active) return;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = kWaveM * wave + 16 * mt + 4 * (lane >> 4) + r;
      if (m >= m_cnt) continue;
      const size_t pos = (size_t)(m_first + m);
      if (SWIGLU) {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const int n = n0 + 16 * nt + (lane & 15);
          if (n >= f) continue;
          const float a = acc[mt][nt][r], c = acc[mt][nt + 4][r];
          ((uint16_t*)out)[pos * out_ld + n] = f2bf(silu(a) * c);
        }
      } else {
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
          const int n = n0 + 16 * nt + (lane & 15);
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

// out[t][c] = sum_i w[t][i] * y[slot_of[t*k+i]][c] (+ the shared expert's
// output, the sum of its ys_parts partial planes), i ascending.
template <typename TOUT>
__global__ void combine_kernel(const float* __restrict__ y, const float* __restrict__ ys,
                               int ys_parts, size_t ys_split, const float* __restrict__ topk_w,
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
  if (ys) {
    // the shared expert's reduction parts, summed in order
    float sh = 0.0f;
    for (int z = 0; z < ys_parts; ++z) sh += ys[(size_t)z * ys_split + (size_t)t * d + c];
    acc += sh;
  }
  if constexpr (sizeof(TOUT) == 2)
    out[(size_t)t * d + c] = f2bf(acc);
  else
    out[(size_t)t * d + c] = acc;
}

// Chunk table of one (expert, bit-width) bucket: positions m_first .. +cnt
// in chunks of at most kChunk (the streamed forward computes one bucket per
// launch pair).
__global__ void unit_chunks_kernel(int m_first, int cnt, int bits, int expert, int n_ub,
                                   int32_t* __restrict__ chunks) {
  for (int c = threadIdx.x; c < n_ub; c += blockDim.x) {
    const int m0 = c * kChunk;
    chunks[4 * c] = m_first + m0;
    chunks[4 * c + 1] = m0 < cnt ? min(kChunk, cnt - m0) : 0;
    chunks[4 * c + 2] = bits;
    chunks[4 * c + 3] = expert;
  }
}

// Copy the nested delta of expert e from host to device memory: planes
// [from, to) (the bit-widths' planes; from = 0: nothing present), the scale
// levels they add, and the zero points with the first load.  Both buffers are
// in the canonical tiled layout, so every copy is one strided rectangle (one
// row per (row block, group) block).
hipError_t copy_delta(const d2moe_mwq* hm, const d2moe_mwq* dm, int e, int from, int to,
                      hipStream_t io) {
  if (to <= from) return hipSuccess;
  const int BR = 2048 / dm->group, KB = dm->cols / dm->group;
  const size_t nblk = (size_t)(dm->rows / BR) * KB;
  const int levels = dm->b_max - dm->b_min + 1;
  const int p0 = from, p1 = to;
  const size_t ppitch = (size_t)dm->b_max * 256;
  const size_t poff = (size_t)e * nblk * ppitch + (size_t)p0 * 256;
  hipError_t err = hipMemcpy2DAsync((char*)dm->planes + poff, ppitch, (const char*)hm->planes + poff,
                                    ppitch, (size_t)(p1 - p0) * 256, nblk,
                                    hipMemcpyHostToDevice, io);
  if (err != hipSuccess) return err;
  const int l0 = from == 0 ? 0 : from - dm->b_min + 1, l1 = to - dm->b_min + 1;
  const size_t spitch = (size_t)levels * BR * 2;
  const size_t soff = (size_t)e * nblk * spitch + (size_t)l0 * BR * 2;
  err = hipMemcpy2DAsync((char*)dm->scales + soff, spitch, (const char*)hm->scales + soff, spitch,
                         (size_t)(l1 - l0) * BR * 2, nblk, hipMemcpyHostToDevice, io);
  if (err != hipSuccess) return err;
  if (from == 0) {
    const size_t zoff = (size_t)e * nblk * BR;
    err = hipMemcpyAsync(dm->zeros + zoff, hm->zeros + zoff, nblk * BR, hipMemcpyHostToDevice, io);
  }
  return err;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Chunk-table bound for n positions in nb buckets: every nonempty bucket
// contributes one chunk plus one per kChunk positions.
int chunk_bound(int n, int nb) { return (nb < n ? nb : n) + (n + kChunk - 1) / kChunk; }

// The shared expert is one bucket of T positions, so its launches are small:
// its positions are cut into as many equal chunks (multiples of 64, at most
// kChunk) as keep the W1/W3 GEMM within one round of kFillWgs workgroups,
// and its W2 reduction is split into parts until W2 has about as many (each
// part at least 16 steps); the parts' partial sums are added by the
// combine.  A function of the sizes only, so the workspace layout and the
// launches agree.
constexpr int kFillWgs = 256;
void shared_plan(int T, int d, int shared_d_ff, int* cs, int* ksplit) {
  const long tiles13 = (shared_d_ff + kTileRows / 2 - 1) / (kTileRows / 2);
  long nch = kFillWgs / tiles13;
  const long most_ch = (T + kWaveM - 1) / kWaveM;
  nch = nch < 1 ? 1 : (nch > most_ch ? most_ch : nch);
  int c = (int)(((T + nch - 1) / nch + kWaveM - 1) / kWaveM * kWaveM);
  c = c > kChunk ? kChunk : (c < kWaveM ? kWaveM : c);
  *cs = c;
  const long wg2 = (long)((d + kTileRows - 1) / kTileRows) * ((T + c - 1) / c);
  const int steps2 = shared_d_ff / kStepK;
  int sp = (int)((kFillWgs + wg2 - 1) / wg2);
  const int most = steps2 / 16 > 1 ? steps2 / 16 : 1;
  *ksplit = sp < 1 ? 1 : (sp > most ? most : sp);
}

// `split`: run chunks of at most 64 positions in the narrow kernel (worth
// it when most chunks are narrow: a second launch runs after the first, and
// its workgroups are as long as the reduction dimension).  `part` (with
// split): 0 both launches, 1 the wide one only, 2 the narrow one only.
template <bool SWIGLU>
hipError_t run_gemm(const uint16_t* in, int in_ld, const int32_t* perm, int kdiv, const MwqView& W,
                    const int32_t* chunks, int n_ub, int f, void* out, int out_ld, bool split,
                    hipStream_t s, int ksplit = 1, size_t out_split = 0, int part = 0) {
  const int N = SWIGLU ? W.rows / 2 : W.rows;
  const int per = SWIGLU ? kTileRows / 2 : kTileRows;
  // weight-row tiles vary fastest: consecutive workgroups, which the
  // dispatcher deals round-robin to the 8 XCDs, share one chunk, so every
  // XCD's L2 holds the activations of the one or two chunks in flight
  // rather than of all of them
  dim3 grid((N + per - 1) / per, n_ub, SWIGLU ? 1 : ksplit);
  if (n_ub <= 0) return hipSuccess;
  // chunks of more than 64 positions (all of them without split), then the
  // chunks of at most 64
  const int sp = split ? 1 : 0;
  constexpr int kWide = 64 * n_waves<false>(), kNarrow = 64 * n_waves<true>();
  const bool wide = !split || part != 2, narrow = split && part != 1;
  if (W.group == 128) {
    if (wide)
      bgemm_kernel<128, SWIGLU, false><<<grid, kWide, 0, s>>>(in, in_ld, perm, kdiv, W, chunks, f,
                                                              N, out, out_ld, sp, out_split);
    if (narrow)
      bgemm_kernel<128, SWIGLU, true><<<grid, kNarrow, 0, s>>>(in, in_ld, perm, kdiv, W, chunks, f,
                                                               N, out, out_ld, sp, out_split);
  } else {
    if (wide)
      bgemm_kernel<64, SWIGLU, false><<<grid, kWide, 0, s>>>(in, in_ld, perm, kdiv, W, chunks, f,
                                                             N, out, out_ld, sp, out_split);
    if (narrow)
      bgemm_kernel<64, SWIGLU, true><<<grid, kNarrow, 0, s>>>(in, in_ld, perm, kdiv, W, chunks, f,
                                                              N, out, out_ld, sp, out_split);
  }
  return hipGetLastError();
}

}  // namespace

FwdWorkspace fwd_workspace_layout(int T, int d, int d_ff, int E, int k, int shared_d_ff) {
  FwdWorkspace L;
  size_t off = 0;
  // chunk tables of the routed experts (at most 8 bit-widths per expert) and
  // of the shared expert
  L.chunk_n = chunk_bound(T * k, E * 8);
  L.shared_chunk = kChunk;
  L.shared_ksplit = 1;
  if (shared_d_ff > 0) shared_plan(T, d, shared_d_ff, &L.shared_chunk, &L.shared_ksplit);
  L.schunk_n = shared_d_ff > 0 ? (T + L.shared_chunk - 1) / L.shared_chunk : 0;
  L.sched_off = off;  off += align256(sizeof(int32_t) * 4 * (size_t)(L.chunk_n + L.schunk_n));
  L.h_off = off;      off += align256(sizeof(uint16_t) * (size_t)T * k * d_ff);
  L.hs_off = off;     off += align256(sizeof(uint16_t) * (size_t)T * shared_d_ff);
  L.y_off = off;      off += align256(sizeof(float) * (size_t)T * k * d);
  L.ys_off = off;
  off += align256(sizeof(float) * (size_t)L.shared_ksplit * T * (shared_d_ff > 0 ? d : 0));
  L.xb_off = off;     off += align256(sizeof(uint16_t) * (size_t)T * d);
  const size_t nd = T <= kDecodeMaxTokens ? (size_t)T * k : 0;  // decode positions
  // decode work list: at most one run per active expert plus one per 8 positions
  // (runs of up to 16 positions need fewer)
  L.elist_off = off;  off += align256(sizeof(int32_t) * (4 * ((size_t)E + (nd + 7) / 8) + 4));
  const size_t nz = nd ? nd + 1 : 0;  // plus one all-zero activation slot
  L.xq13_off = off;   off += align256(nz * d * 2);
  const size_t nxs = nz ? nz + 24 : 0;  // info words, padded for 24-position reads
  L.xs13_off = off;   off += align256(nxs * sizeof(uint32_t));
  L.h32_off = off;    off += align256(nd * d_ff * sizeof(float));
  L.xq2_off = off;    off += align256(nz * d_ff * 2);
  L.xs2_off = off;    off += align256(nxs * sizeof(uint32_t));
  // partial maxima of |h|: one word per (position, 16-row block of d_ff)
  L.hmax_off = off;   off += align256(nd * ((size_t)(d_ff + 15) / 16) * sizeof(uint32_t));
  L.total = off;
  return L;
}

// Side streams of the calling host thread on the current device (created at
// its first concurrent forward there, default priority, kept until the
// process ends), and the events that fork work onto them from the caller's
// stream and join it back.  Per thread, so that calls from different host
// threads never wait on each other's events.
struct SideStreams {
  hipStream_t s[2] = {nullptr, nullptr};
  hipEvent_t fork = nullptr, join[2] = {nullptr, nullptr};
};
constexpr int kMaxSideDevices = 64;
hipError_t side_streams(SideStreams** out) {
  thread_local SideStreams cache[kMaxSideDevices];
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxSideDevices) return hipErrorInvalidDevice;
  SideStreams& ss = cache[dev];
  if (ss.fork == nullptr) {
    SideStreams n;
    for (int i = 0; i < 2; ++i) {
      if ((err = hipStreamCreateWithFlags(&n.s[i], hipStreamNonBlocking)) != hipSuccess) return err;
      if ((err = hipEventCreateWithFlags(&n.join[i], hipEventDisableTiming)) != hipSuccess)
        return err;
    }
    if ((err = hipEventCreateWithFlags(&n.fork, hipEventDisableTiming)) != hipSuccess) return err;
    ss = n;
  }
  *out = &ss;
  return hipSuccess;
}

// The layer with its expert weights streamed in (Sec. 3.4): units in the
// given order; each unit's nested delta is copied on `io`, and the unit's
// bucket is computed on `s` once that copy has landed (an event per unit), so
// the copy of the next unit overlaps the computation of this one.  The
// per-position arithmetic is that of the grouped GEMM path of
// launch_forward (same chunking of a bucket, same narrow/wide split).
hipError_t launch_forward_streamed(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E,
                                   int k, const d2moe_mwq* hw13, const d2moe_mwq* hw2,
                                   const d2moe_mwq* w13, const d2moe_mwq* w2, uint8_t* resident,
                                   const d2moe_routing* r, const int32_t* hist_host,
                                   const d2moe_unit* units, int n_units, void* out, void* ws,
                                   hipStream_t s, hipStream_t io, const hipEvent_t* events) {
  const FwdWorkspace L = fwd_workspace_layout(T, d, d_ff, E, k, 0);
  char* base = (char*)ws;
  const int Lv = w13->b_max - w13->b_min + 1, b_min = w13->b_min;
  int32_t* chunks = (int32_t*)(base + L.sched_off);
  uint16_t* h = (uint16_t*)(base + L.h_off);
  float* y = (float*)(base + L.y_off);
  hipError_t err;
  const uint16_t* xb = (const uint16_t*)x;
  if (T > 0 && xd == D2MOE_F32) {
    uint16_t* xw = (uint16_t*)(base + L.xb_off);
    const size_t n = (size_t)T * d;
    to_bf16_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>((const float*)x, n, xw);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    xb = xw;
  }
  // bucket offsets from the host counts (exclusive scan, expert major)
  int off[64 * 8 + 1];
  off[0] = 0;
  for (int i = 0; i < E * Lv; ++i) off[i + 1] = off[i] + hist_host[i];
  const MwqView W13 = view_of(w13), W2 = view_of(w2);
  const bool split = (long)T * k <= 64L * E;
  for (int i = 0; i < n_units; ++i) {
    const d2moe_unit& u = units[i];
    if ((err = copy_delta(hw13, w13, u.expert, u.load_from, u.load_to, io)) != hipSuccess)
      return err;
    if ((err = copy_delta(hw2, w2, u.expert, u.load_from, u.load_to, io)) != hipSuccess)
      return err;
    if ((err = hipEventRecord(events[i], io)) != hipSuccess) return err;
    if ((err = hipStreamWaitEvent(s, events[i], 0)) != hipSuccess) return err;
    if (resident[u.expert] < u.load_to) resident[u.expert] = (uint8_t)u.load_to;
    if (u.count <= 0) continue;
    const int m_first = off[u.expert * Lv + (u.bits - b_min)];
    const int n_ub = (u.count + kChunk - 1) / kChunk;
    unit_chunks_kernel<<<1, 64, 0, s>>>(m_first, u.count, u.bits, u.expert, n_ub, chunks);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    err = run_gemm<true>(xb, d, r->perm, k, W13, chunks, n_ub, d_ff, h, d_ff, split, s);
    if (err != hipSuccess) return err;
    err = run_gemm<false>(h, d_ff, nullptr, 1, W2, chunks, n_ub, d_ff, y, d, split, s);
    if (err != hipSuccess) return err;
  }
  if (T == 0) return hipSuccess;
  dim3 cg((d + 255) / 256, T);
  if (xd == D2MOE_BF16)
    combine_kernel<uint16_t><<<cg, 256, 0, s>>>(y, nullptr, 1, 0, r->topk_w, r->slot_of, k, d,
                                                (uint16_t*)out);
  else
    combine_kernel<float><<<cg, 256, 0, s>>>(y, nullptr, 1, 0, r->topk_w, r->slot_of, k, d,
                                             (float*)out);
  return hipGetLastError();
}

hipError_t launch_forward(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                          const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                          const d2moe_mwq* sw13, const d2moe_mwq* sw2, int shared_bits,
                          int shared_d_ff, void* out, void* ws, hipStream_t s,
                          const hipEvent_t* events, bool concurrent) {
  if (T == 0) return hipSuccess;
  const bool has_shared = sw13 != nullptr;
  const FwdWorkspace L = fwd_workspace_layout(T, d, d_ff, E, k, has_shared ? shared_d_ff : 0);
  char* base = (char*)ws;
  const int Lv = w13->b_max - w13->b_min + 1;
  const int nb = E * Lv;
  int32_t* chunks = (int32_t*)(base + L.sched_off);
  int32_t* schunks = chunks + 4 * (size_t)L.chunk_n;
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
  // Concurrency: the shared expert's chain, and with split the narrow
  // routed chunks, run on side streams forked from `s` (they write disjoint
  // workspace: hs / ys, and other rows of h / y than the wide chunks); the
  // combine waits for both.  Not with events: those time the kernels on `s`.
  // (Running every other chunk of a layer without split, such as a
  // 2048-token prefill, beside the rest measured 4 % slower: the two W1/W3
  // launches contend rather than fill each other's tails.)
  const bool decode = decode_path_ok(w13, w2, T);
  const bool split = !decode && (long)T * k <= 64L * E;
  const bool fork_shared = concurrent && !events && has_shared;
  const bool fork_narrow = concurrent && !events && split;
  SideStreams* side = nullptr;
  if (fork_shared || fork_narrow)
    if ((err = side_streams(&side)) != hipSuccess) return err;

  if (has_shared) {
    hipStream_t ss = s;
    if (fork_shared) {
      ss = side->s[1];
      if ((err = hipEventRecord(side->fork, s)) != hipSuccess) return err;
      if ((err = hipStreamWaitEvent(ss, side->fork, 0)) != hipSuccess) return err;
    }
    const int ns_ub = L.schunk_n, cs = L.shared_chunk, ks = L.shared_ksplit;
    chunk_kernel<<<1, kChunkThreads, 0, ss>>>(nullptr, nullptr, 0, 1, sw13->b_min, T, shared_bits,
                                             cs, ns_ub, schunks);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const MwqView S13 = view_of(sw13), S2 = view_of(sw2);
    err = run_gemm<true>(xb, d, nullptr, 1, S13, schunks, ns_ub, shared_d_ff, hs, shared_d_ff,
                         cs <= kWaveM, ss);
    if (err != hipSuccess) return err;
    err = run_gemm<false>(hs, shared_d_ff, nullptr, 1, S2, schunks, ns_ub, shared_d_ff, ys, d,
                          cs <= kWaveM, ss, ks, (size_t)T * d);
    if (err != hipSuccess) return err;
    if (fork_shared && (err = hipEventRecord(side->join[1], ss)) != hipSuccess) return err;
  }

  if (decode) {
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
    const int n_ub = chunk_bound(T * k, nb);
    chunk_kernel<<<1, kChunkThreads, 0, s>>>(r->hist, r->offsets, nb, Lv, w13->b_min, 0, 0,
                                            kChunk, n_ub, chunks);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const MwqView W13 = view_of(w13), W2 = view_of(w2);
    // narrow chunks get their own launch when experts average at most 64
    // positions; forked, they run beside the wide ones
    if (fork_narrow) {
      hipStream_t sn = side->s[0];
      if ((err = hipEventRecord(side->fork, s)) != hipSuccess) return err;
      if ((err = hipStreamWaitEvent(sn, side->fork, 0)) != hipSuccess) return err;
      err = run_gemm<true>(xb, d, r->perm, k, W13, chunks, n_ub, d_ff, h, d_ff, true, sn, 1, 0, 2);
      if (err != hipSuccess) return err;
      err = run_gemm<false>(h, d_ff, nullptr, 1, W2, chunks, n_ub, d_ff, y, d, true, sn, 1, 0, 2);
      if (err != hipSuccess) return err;
      if ((err = hipEventRecord(side->join[0], sn)) != hipSuccess) return err;
    }
    const int part = fork_narrow ? 1 : 0;
    if (events && (err = hipEventRecord(events[0], s)) != hipSuccess) return err;
    err = run_gemm<true>(xb, d, r->perm, k, W13, chunks, n_ub, d_ff, h, d_ff, split, s, 1, 0, part);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[1], s)) != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[2], s)) != hipSuccess) return err;
    err = run_gemm<false>(h, d_ff, nullptr, 1, W2, chunks, n_ub, d_ff, y, d, split, s, 1, 0, part);
    if (err != hipSuccess) return err;
    if (events && (err = hipEventRecord(events[3], s)) != hipSuccess) return err;
    if (fork_narrow && (err = hipStreamWaitEvent(s, side->join[0], 0)) != hipSuccess) return err;
  }
  if (fork_shared && (err = hipStreamWaitEvent(s, side->join[1], 0)) != hipSuccess) return err;

  dim3 cg((d + 255) / 256, T);
  if (xd == D2MOE_BF16)
    combine_kernel<uint16_t><<<cg, 256, 0, s>>>(y, has_shared ? ys : nullptr, L.shared_ksplit,
                                                (size_t)T * d, r->topk_w, r->slot_of, k, d,
                                                (uint16_t*)out);
  else
    combine_kernel<float><<<cg, 256, 0, s>>>(y, has_shared ? ys : nullptr, L.shared_ksplit,
                                             (size_t)T * d, r->topk_w, r->slot_of, k, d,
                                             (float*)out);
  return hipGetLastError();
}

}  // namespace d2moe
