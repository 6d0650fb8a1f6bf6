/*
 * CPU oracle for the D^2MoE MoE-layer hot path (dual routing + matryoshka
 * weight quantization).  TEST INFRASTRUCTURE ONLY: the tests, the smoke check
 * and the benchmark's CPU-baseline leg may call it; the product library never
 * links or calls it, and it shares no code with the GPU path.
 *
 * Plain, single-threaded, slow on purpose.  Every function states the passage
 * of the paper it follows.  Quantization decisions (codes, signs, scales) are
 * taken in IEEE binary32 with no FMA contraction, because the packed codes are
 * integers that the GPU must reproduce bit for bit; everything that produces a
 * floating-point result (logits, softmax, expert FFN, combine) is computed in
 * binary64.
 *
 * Conventions shared with the canonical packed format (a definition, not code):
 *   - a weight matrix W is [rows][cols], groups of `group` consecutive columns
 *     (the reduction dimension) share quantization parameters;
 *   - bit-width ladder b_min = b1 ... b_max = bK, one bit per step;
 *   - level 0 holds the base scale s_b1, level l >= 1 the residual scale of
 *     bit-width b1 + l;  levels = b_max - b_min + 1;
 *   - plane p < b1 holds bit p of the base code Q_b1; plane p >= b1 holds the
 *     residual sign of bit-width p + 1 (1 = +1, 0 = -1); a b-bit read uses
 *     planes 0 .. b-1.
 */
#ifndef D2MOE_ORACLE_H
#define D2MOE_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* IEEE binary32 -> binary16, round to nearest even (with subnormals/inf). */
uint16_t oracle_f32_to_f16(float f);
float oracle_f16_to_f32(uint16_t h);
/* IEEE binary32 -> bfloat16 (round to nearest even), returned widened. */
float oracle_round_bf16(float f);

/* MWQ logical quantization of one matrix (Sec. 3.3.1, Eq. 2-5, Algorithm 1
 * read with X = I).  Outputs:
 *   q1     [rows][cols]                 base code Q_b1 in [0, 2^b_min - 1]
 *   zeros  [rows][cols/group]           integer zero point z_b1
 *   scales [levels][rows][cols/group]   binary16 bit patterns
 *   signs  [b_max-b_min][rows][cols]    residual sign bits (1 = +1)
 *   resid_sq (optional, may be NULL) [levels][rows][cols/group]: sum of
 *          squared fp32 residuals after each level (level 0 = after base).
 * Returns 0, or -1 on invalid arguments. */
int oracle_mwq_quantize(const float* W, int rows, int cols, int group,
                        int b_min, int b_max, uint8_t* q1, uint8_t* zeros,
                        uint16_t* scales, uint8_t* signs, double* resid_sq);

/* Calibration-aware MWQ of one matrix (Sec. 3.3.1, Eq. 3 and Eq. 5 with
 * calibration activations X; Algorithm 1's block-level error compensation).
 * U: [cols][cols] binary32, the upper Cholesky factor of (2 X X^T + lambda I)^-1
 * (upper triangle read); gamma: columns per compensation block, a multiple
 * of group dividing cols.  Outputs as oracle_mwq_quantize (no resid_sq);
 * targets (optional) [levels][rows][cols]: the value each column had when
 * its block was quantized at that level (weights at level 0, residuals of
 * the lower levels above).  With U diagonal the codes equal
 * oracle_mwq_quantize's.  Returns 0, or -1 on invalid arguments. */
int oracle_mwq_quantize_calibrated(const float* W, int rows, int cols, int group,
                                   int b_min, int b_max, const float* U, int gamma,
                                   uint8_t* q1, uint8_t* zeros, uint16_t* scales,
                                   uint8_t* signs, float* targets);

/* Dequantized weights at bit-width b (Eq. 2 and the nested sum under Eq. 5),
 * exact in binary64. */
int oracle_mwq_dequant(int rows, int cols, int group, int b_min, int b_max,
                       int b, const uint8_t* q1, const uint8_t* zeros,
                       const uint16_t* scales, const uint8_t* signs,
                       double* What);

/* Canonical tiled bit-plane layout of one expert matrix (written out from the
 * logical codes).  group must be 64 or 128; rows % (2048/group) == 0.
 *   planes [rows/BR][cols/group][b_max][64] uint32, BR = 2048/group;
 *          word w of a (block, plane): row-in-block w % BR, 32-column
 *          sub-block w / BR, bit j <-> column 32*(w/BR) + j (LSB first);
 *   scales [rows/BR][cols/group][levels][BR] binary16;
 *   zeros  [rows/BR][cols/group][BR] uint8. */
int oracle_mwq_pack(int rows, int cols, int group, int b_min, int b_max,
                    const uint8_t* q1, const uint8_t* zeros,
                    const uint16_t* scales, const uint8_t* signs,
                    uint32_t* planes, uint16_t* scales_out,
                    uint8_t* zeros_out);

/* Gate logits (expert router of the dual routing, Fig. 1), binary64
 * accumulation in ascending column order, plus optional bias. */
int oracle_gate_logits(const float* x, int T, int d, const float* Wg,
                       const float* bias, int E, double* logits);

/* Dual routing from logits: top-k experts per token (largest logit first,
 * ties to the lower expert index), softmax over the k selected logits,
 * bit-width lookup bit_table[token_req[t]][expert], the (expert, bit-width)
 * selection counts B_{j,k} of Sec. 3.4.3, their exclusive scan (expert major,
 * bit minor), the stable permutation of the T*k (token, slot) pairs by that
 * key, its inverse, and the largest bit-width requested per expert (0 if
 * none).  Returns 0, -1 on invalid arguments, -2 if a table entry or request
 * index is out of range. */
int oracle_route_from_logits(const double* logits, int T, int E, int k,
                             const int* token_req, const uint8_t* bit_table,
                             int R, int b_min, int b_max, int* topk_idx,
                             double* topk_w, uint8_t* topk_bits, int* hist,
                             int* offsets, int* perm, int* slot_of,
                             uint8_t* maxbit);

/* One SwiGLU expert at bit-width b from logical codes, for n input vectors:
 *   a = W1_b x, c = W3_b x, h = silu(a) * c, y = W2_b h     (binary64)
 * w13 codes describe a [2f][d] matrix (W1 rows then W3 rows); w2 codes a
 * [d_out][f] matrix: all d rows of W2, or any subset of its rows, since MWQ
 * codes of a row depend on that row alone.  x is [n][d] binary64, y is
 * [n][d_out]. */
int oracle_expert_ffn(int d, int f, int d_out, int group13, int group2, int b_min,
                      int b_max, int b,
                      const uint8_t* q1_13, const uint8_t* zeros_13,
                      const uint16_t* scales_13, const uint8_t* signs_13,
                      const uint8_t* q1_2, const uint8_t* zeros_2,
                      const uint16_t* scales_2, const uint8_t* signs_2,
                      const double* x, int n, double* y);

/* Weighted combine: out[t] = sum_i w[t,i] * y[slot t*k+i] in i order. */
int oracle_combine(int T, int k, int d, const double* topk_w,
                   const double* y_slot, double* out);

/* RMS normalisation with unit weight, binary64, as applied to the hidden
 * state before each MoE layer of the decoders of Sec. 5.1:
 * h[t][c] = x[t][c] / sqrt(mean_c x[t][c]^2 + eps), sums in ascending c. */
int oracle_rmsnorm(int T, int d, double eps, const double* x, double* h);

#ifdef __cplusplus
}
#endif
#endif
