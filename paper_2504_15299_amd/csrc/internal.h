// Internal declarations shared by the HIP translation units of libd2moe.
// Layout helpers for the canonical tiled bit-plane MWQ format and the
// host-side launchers each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/d2moe.h"

namespace d2moe {

// ---- canonical layout -----------------------------------------------------
// A block is BR = 2048/group rows x group columns; per (block, plane) there are
// 64 uint32 words; word w covers row w % BR and columns 32*(w/BR) .. +31.
__host__ __device__ inline int block_rows(int group) { return 2048 / group; }

struct MwqView {
  int E, rows, cols, group, b_min, b_max;
  const uint32_t* planes;
  const uint16_t* scales;
  const uint8_t* zeros;
  __host__ __device__ int BR() const { return 2048 / group; }
  __host__ __device__ int KB() const { return cols / group; }
  __host__ __device__ int levels() const { return b_max - b_min + 1; }
  // index of block (row-block rb, column-block kb) of expert e
  __host__ __device__ size_t block(int e, int rb, int kb) const {
    return ((size_t)e * (rows / BR()) + rb) * KB() + kb;
  }
  __host__ __device__ size_t plane_word(size_t blk, int p, int w) const {
    return (blk * b_max + p) * 64 + w;
  }
  __host__ __device__ size_t scale_idx(size_t blk, int lev, int i) const {
    return (blk * levels() + lev) * BR() + i;
  }
  __host__ __device__ size_t zero_idx(size_t blk, int i) const {
    return blk * BR() + i;
  }
};

inline MwqView view_of(const d2moe_mwq* m) {
  MwqView v;
  v.E = m->n_experts; v.rows = m->rows; v.cols = m->cols; v.group = m->group;
  v.b_min = m->b_min; v.b_max = m->b_max;
  v.planes = m->planes; v.scales = m->scales; v.zeros = m->zeros;
  return v;
}

// Binary16 bit pattern <-> float (hardware conversions; float -> binary16
// rounds to nearest even, subnormals kept).
__device__ inline float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
__device__ inline uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

// bf16 helpers (round to nearest even).
__device__ inline uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ inline float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// ---- launchers (return hipError_t of the launch) ---------------------------
hipError_t launch_pack(const float* W, const d2moe_mwq* out, hipStream_t s);
hipError_t launch_debug_unpack(const d2moe_mwq* w, int expert, int bits, uint8_t* q1,
                               int8_t* signs, hipStream_t s);
hipError_t launch_route(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                        const float* bias, int E, int k, const int32_t* token_req,
                        const uint8_t* bit_table, int R, int b_min, int b_max,
                        const d2moe_routing* out, hipStream_t s);
hipError_t launch_route_learned(const void* x, d2moe_dtype xd, int T, int d, const float* Wg,
                                const float* bias, int E, int k, const float* Wr,
                                const float* br, int b_min, int b_max, float* bit_logits,
                                const d2moe_routing* out, hipStream_t s);

// Forward workspace layout (256-byte aligned sub-buffers).  The decode
// buffers exist only when T <= kDecodeMaxTokens.
constexpr int kDecodeMaxTokens = 64;
struct FwdWorkspace {
  size_t sched_off, h_off, hs_off, y_off, ys_off, xb_off;
  size_t elist_off, xq13_off, xs13_off, h32_off, xq2_off, xs2_off, hmax_off;
  size_t total;
  int chunk_n, schunk_n;  // grouped-GEMM chunk-table entries (routed, shared)
  int shared_chunk;       // positions per chunk of the shared expert
  int shared_ksplit;      // parts of the shared W2 reduction (partial sums summed by combine)
};

struct DecodeBuffers {
  int32_t* elist;   // [work items][4]
  uint8_t *xq13, *xq2;
  uint32_t *xs13, *xs2;  // [T*k+1] position info words
  float* h32;       // [T*k][d_ff]
  uint32_t* hmax;   // [T*k][d_ff/16] largest |h| of each position per 16-row block (binary32 bits)
  float* y;         // [T*k][d]
};

bool decode_path_ok(const d2moe_mwq* w13, const d2moe_mwq* w2, int T);
hipError_t launch_decode_ffn(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                             const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                             const DecodeBuffers& b, hipStream_t s, const hipEvent_t* events);
FwdWorkspace fwd_workspace_layout(int T, int d, int d_ff, int E, int k, int shared_d_ff);

hipError_t launch_forward_streamed(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E,
                                   int k, const d2moe_mwq* hw13, const d2moe_mwq* hw2,
                                   const d2moe_mwq* w13, const d2moe_mwq* w2, uint8_t* resident,
                                   const d2moe_routing* r, const int32_t* hist_host,
                                   const d2moe_unit* units, int n_units, void* out, void* ws,
                                   hipStream_t s, hipStream_t io, const hipEvent_t* events);
int norm_max_cols();
int hebf_order(const int32_t* hist, int E, int b_min, int b_max, const uint8_t* resident,
               d2moe_unit* units);
int budget_plan(const uint8_t* want, int n_layers, int E, const int64_t* level_bytes, int K,
                int64_t budget, uint8_t* res, d2moe_budget_action* actions, int max_actions);
size_t calib_factor_workspace(int n);
hipError_t launch_calib_factor(const float* X, int tokens, int n, double lambda, float* U,
                               void* ws, int32_t* info, hipStream_t s);
size_t calib_pack_workspace(int rows, int cols, int gamma);
hipError_t launch_pack_calibrated(const float* W, const float* U, int gamma,
                                  const d2moe_mwq* out, void* ws, hipStream_t s);
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int blocks,
                              hipStream_t s);
hipError_t launch_residual_rmsnorm(float* x, const void* y, d2moe_dtype yd, int T, int d,
                                   float eps, void* h, d2moe_dtype hd, hipStream_t s);

// concurrent: independent parts of the layer (the shared expert, the
// narrow routed chunks) may run on this host thread's side streams of the
// current device, forked from and joined back to `s` with events.
hipError_t launch_forward(const void* x, d2moe_dtype xd, int T, int d, int d_ff, int E, int k,
                          const d2moe_mwq* w13, const d2moe_mwq* w2, const d2moe_routing* r,
                          const d2moe_mwq* sw13, const d2moe_mwq* sw2, int shared_bits,
                          int shared_d_ff, void* out, void* ws, hipStream_t s,
                          const hipEvent_t* events, bool concurrent);

}  // namespace d2moe
