/*
 * CPU oracle for the D^2MoE MoE-layer hot path.  TEST INFRASTRUCTURE ONLY
 * (tests, smoke check, benchmark CPU-baseline leg); the product library never
 * links or calls it.  See oracle.h for the conventions.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC oracle.c -lm
 * (binary32 steps must not be fused or reassociated: the quantizer's integer
 * decisions are compared bit for bit with the GPU's).
 *
 * Readings of the paper taken here (each is listed with its reason in the
 * design notes):
 *  - Eq. 3 and Eq. 5 minimise ||WX - W^X||^2 over calibration activations X
 *    that are not available; X = I is used.  With X = I the Hessian of
 *    Algorithm 1 is a multiple of I, its Cholesky factor is diagonal, the
 *    off-diagonal block used for the block compensation is zero, and
 *    Algorithm 1 reduces to independent per-group quantization.
 *  - Base level (Eq. 2): asymmetric min-max with 0 inside the range, scale
 *    stored as binary16, integer zero point, round half to even, codes
 *    clamped to [0, 2^b1 - 1].
 *  - Residual level (Eq. 4-5): the one-bit code is the sign of the residual
 *    (sign(0) = +1) and the scale is the mean absolute residual over the
 *    group, which is the exact least-squares scale of a sign code at X = I;
 *    stored as binary16, and the quantizer continues from the stored value.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---- number formats (IEEE 754 definitions) ---------------------------- */

/* binary32 -> binary16, round to nearest, ties to even.  Works in binary64,
 * where every scaling by a power of two below is exact. */
uint16_t oracle_f32_to_f16(float f) {
  uint32_t bits;
  memcpy(&bits, &f, 4);
  uint16_t sign = (uint16_t)((bits >> 16) & 0x8000u);
  if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
  double v = fabs((double)f);
  if (isinf(f)) return (uint16_t)(sign | 0x7c00u);
  if (v < ldexp(1.0, -14)) {
    /* subnormal range: value = q * 2^-24, q in [0, 1024]; q == 1024 is the
     * smallest normal number and encodes the same way */
    double q = nearbyint(v * ldexp(1.0, 24));
    return (uint16_t)(sign | (uint16_t)q);
  }
  int ex;
  frexp(v, &ex);           /* v = m * 2^ex, m in [0.5, 1) */
  int e = ex - 1;          /* v in [2^e, 2^(e+1)) */
  double q = nearbyint(v * ldexp(1.0, 10 - e)); /* in [1024, 2048] */
  if (q >= 2048.0) {
    q = 1024.0;
    e += 1;
  }
  if (e > 15) return (uint16_t)(sign | 0x7c00u);
  return (uint16_t)(sign | (uint16_t)((e + 15) << 10) | (uint16_t)(q - 1024.0));
}

float oracle_f16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int m = h & 0x3ff;
  double v;
  if (e == 0)
    v = ldexp((double)m, -24);
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = ldexp((double)(m + 1024), e - 25);
  return (float)(sign ? -v : v);
}

float oracle_round_bf16(float f) {
  if (isnan(f)) return f;
  uint32_t bits;
  memcpy(&bits, &f, 4);
  /* keep the top 16 bits, round to nearest even on the dropped 16 */
  uint32_t lower = bits & 0xffffu;
  uint32_t upper = bits & 0xffff0000u;
  int round_up = (lower > 0x8000u) || (lower == 0x8000u && (upper & 0x10000u));
  if (round_up) upper += 0x10000u; /* carries into the exponent correctly */
  float out;
  memcpy(&out, &upper, 4);
  return out;
}

/* ---- MWQ quantization (Sec. 3.3.1) ------------------------------------ */

static int check_ladder(int b_min, int b_max) {
  return b_min >= 1 && b_min <= b_max && b_max <= 8;
}

int oracle_mwq_quantize(const float* W, int rows, int cols, int group,
                        int b_min, int b_max, uint8_t* q1, uint8_t* zeros,
                        uint16_t* scales, uint8_t* signs, double* resid_sq) {
  if (!W || !q1 || !zeros || !scales || rows <= 0 || cols <= 0 ||
      group <= 0 || cols % group != 0 || !check_ladder(b_min, b_max))
    return -1;
  if (b_max > b_min && !signs) return -1;
  const int ng = cols / group;
  const int levels = b_max - b_min + 1;
  const int qmax = (1 << b_min) - 1;
  float* R = (float*)malloc(sizeof(float) * (size_t)group);
  if (!R) return -1;

  for (int n = 0; n < rows; ++n) {
    for (int G = 0; G < ng; ++G) {
      const float* w = W + (size_t)n * cols + (size_t)G * group;
      const size_t gi = (size_t)n * ng + G;

      /* Base level, Eq. 2 with the min-max reading of Eq. 3. */
      float mn = 0.0f, mx = 0.0f;
      for (int k = 0; k < group; ++k) {
        if (w[k] < mn) mn = w[k];
        if (w[k] > mx) mx = w[k];
      }
      float range = mx - mn;
      float s_raw = range / (float)qmax;
      uint16_t s_h = oracle_f32_to_f16(s_raw);
      float s1 = oracle_f16_to_f32(s_h);
      if (!(s1 > 0.0f) || isinf(s1)) {
        /* all-zero group (or overflow): any positive scale reproduces it */
        s_h = 0x3c00u; /* 1.0 */
        s1 = 1.0f;
      }
      float zf = rintf(-mn / s1);
      if (zf < 0.0f) zf = 0.0f;
      if (zf > (float)qmax) zf = (float)qmax;
      const int z = (int)zf;
      zeros[gi] = (uint8_t)z;
      scales[gi] = s_h; /* level 0 */

      double ss = 0.0;
      for (int k = 0; k < group; ++k) {
        float qf = rintf(w[k] / s1 + (float)z);
        if (qf < 0.0f) qf = 0.0f;
        if (qf > (float)qmax) qf = (float)qmax;
        const int q = (int)qf;
        q1[(size_t)n * cols + (size_t)G * group + k] = (uint8_t)q;
        const float what = (float)(q - z) * s1;
        R[k] = w[k] - what;
        ss += (double)R[k] * (double)R[k];
      }
      if (resid_sq) resid_sq[gi] = ss;

      /* Residual levels, Eq. 4-5: one sign plane and one scale per bit. */
      for (int lev = 1; lev < levels; ++lev) {
        float acc = 0.0f;
        for (int k = 0; k < group; ++k) acc = acc + fabsf(R[k]);
        const float s_mean = acc / (float)group;
        const uint16_t sb_h = oracle_f32_to_f16(s_mean);
        const float sb = oracle_f16_to_f32(sb_h);
        scales[(size_t)lev * rows * ng + gi] = sb_h;
        uint8_t* sg = signs + (size_t)(lev - 1) * rows * cols +
                      (size_t)n * cols + (size_t)G * group;
        ss = 0.0;
        for (int k = 0; k < group; ++k) {
          const int pos = R[k] >= 0.0f; /* -0.0 >= 0 holds: sign +1 */
          sg[k] = (uint8_t)pos;
          R[k] = pos ? (R[k] - sb) : (R[k] + sb);
          ss += (double)R[k] * (double)R[k];
        }
        if (resid_sq) resid_sq[(size_t)lev * rows * ng + gi] = ss;
      }
    }
  }
  free(R);
  return 0;
}

/* ---- calibration-aware MWQ (Sec. 3.3.1, Eq. 3 and Eq. 5 with calibration
 * activations; Algorithm 1's block compensation) ------------------------
 *
 * Algorithm 1 quantizes W block by block (gamma columns at a time) and, as
 * GPTQ does, moves each block's quantization error onto the columns not yet
 * quantized, weighted by the inverse Hessian of the calibration inputs; the
 * text keeps only this block-level compensation and drops GPTQ's
 * column-by-column corrections inside a block.  With U the upper Cholesky
 * factor of H^-1, H = 2 X X^T + lambda I (so H^-1 = U^T U), the error D_B of
 * block B is carried to the later columns F as
 *     E = D_B U_BB^-1,      T_F <- T_F - E U_BF,
 * which is the least-squares optimal change of T_F for the error D_B
 * ((H^-1)_BB^-1 (H^-1)_BF = U_BB^-1 U_BF).
 * Each bit-width level is one such pass over the blocks, restarting from the
 * uncompensated quantity of that level, with every lower level fixed:
 *   level 0 (Eq. 2): T = W, the block's base codes come from the current T_B
 *     (same per-group rule as oracle_mwq_quantize), D_B = T_B - W^_b1,B;
 *   level l >= 1 (Eq. 4-5): T = R, the residual W - W^ of the levels below
 *     (kept as a chain, updated after each level exactly as in
 *     oracle_mwq_quantize), the block's signs and scales come from the
 *     current T_B, D_B = T_B - s sigma.
 * With U diagonal (X = I) no compensation happens and the codes equal
 * oracle_mwq_quantize's bit for bit.  The integer decisions are taken on
 * binary32 values, as on the GPU; the compensation is written with fmaf in
 * ascending index order so that it has one defined rounding sequence. */
static void base_group(const float* w, int group, int qmax, uint8_t* q,
                       uint8_t* z_out, uint16_t* s_out, float* what) {
  float mn = 0.0f, mx = 0.0f;
  for (int k = 0; k < group; ++k) {
    if (w[k] < mn) mn = w[k];
    if (w[k] > mx) mx = w[k];
  }
  const float range = mx - mn;
  uint16_t s_h = oracle_f32_to_f16(range / (float)qmax);
  float s1 = oracle_f16_to_f32(s_h);
  if (!(s1 > 0.0f) || isinf(s1)) {
    s_h = 0x3c00u;
    s1 = 1.0f;
  }
  float zf = rintf(-mn / s1);
  if (zf < 0.0f) zf = 0.0f;
  if (zf > (float)qmax) zf = (float)qmax;
  const int z = (int)zf;
  *z_out = (uint8_t)z;
  *s_out = s_h;
  for (int k = 0; k < group; ++k) {
    float qf = rintf(w[k] / s1 + (float)z);
    if (qf < 0.0f) qf = 0.0f;
    if (qf > (float)qmax) qf = (float)qmax;
    q[k] = (uint8_t)(int)qf;
    what[k] = (float)((int)qf - z) * s1;
  }
}

int oracle_mwq_quantize_calibrated(const float* W, int rows, int cols, int group,
                                   int b_min, int b_max, const float* U, int gamma,
                                   uint8_t* q1, uint8_t* zeros, uint16_t* scales,
                                   uint8_t* signs, float* targets) {
  if (!W || !U || !q1 || !zeros || !scales || rows <= 0 || cols <= 0 ||
      group <= 0 || cols % group != 0 || gamma <= 0 || gamma % group != 0 ||
      cols % gamma != 0 || !check_ladder(b_min, b_max))
    return -1;
  if (b_max > b_min && !signs) return -1;
  const int ng = cols / group;
  const int levels = b_max - b_min + 1;
  const int qmax = (1 << b_min) - 1;
  float* T = (float*)malloc(sizeof(float) * (size_t)cols);
  float* R = (float*)malloc(sizeof(float) * (size_t)cols);
  float* what = (float*)malloc(sizeof(float) * (size_t)cols);
  float* D = (float*)malloc(sizeof(float) * (size_t)gamma);
  float* E = (float*)malloc(sizeof(float) * (size_t)gamma);
  if (!T || !R || !what || !D || !E) {
    free(T); free(R); free(what); free(D); free(E);
    return -1;
  }
  for (int n = 0; n < rows; ++n) {
    const float* w = W + (size_t)n * cols;
    for (int lev = 0; lev < levels; ++lev) {
      for (int c = 0; c < cols; ++c) T[c] = lev == 0 ? w[c] : R[c];
      for (int b0 = 0; b0 < cols; b0 += gamma) {
        if (targets)
          for (int c = b0; c < b0 + gamma; ++c)
            targets[((size_t)lev * rows + n) * cols + c] = T[c];
        /* quantize the block from its current values */
        for (int G = b0 / group; G < (b0 + gamma) / group; ++G) {
          const size_t gi = (size_t)n * ng + G;
          const int c0 = G * group;
          if (lev == 0) {
            base_group(T + c0, group, qmax, q1 + (size_t)n * cols + c0, zeros + gi,
                       scales + gi, what + c0);
            for (int k = 0; k < group; ++k) D[c0 - b0 + k] = T[c0 + k] - what[c0 + k];
          } else {
            float acc = 0.0f;
            for (int k = 0; k < group; ++k) acc = acc + fabsf(T[c0 + k]);
            const uint16_t sb_h = oracle_f32_to_f16(acc / (float)group);
            const float sb = oracle_f16_to_f32(sb_h);
            scales[(size_t)lev * rows * ng + gi] = sb_h;
            uint8_t* sg = signs + (size_t)(lev - 1) * rows * cols + (size_t)n * cols + c0;
            for (int k = 0; k < group; ++k) {
              const int pos = T[c0 + k] >= 0.0f; /* -0.0 >= 0: sign +1 */
              sg[k] = (uint8_t)pos;
              D[c0 - b0 + k] = pos ? (T[c0 + k] - sb) : (T[c0 + k] + sb);
            }
          }
        }
        /* E = D U_BB^-1 (forward substitution, ascending order) */
        for (int j = 0; j < gamma; ++j) {
          float e = D[j];
          for (int i = 0; i < j; ++i)
            e = fmaf(-E[i], U[(size_t)(b0 + i) * cols + (b0 + j)], e);
          E[j] = e / U[(size_t)(b0 + j) * cols + (b0 + j)];
        }
        /* T_F -= E U_BF */
        for (int f = b0 + gamma; f < cols; ++f) {
          float acc = T[f];
          for (int j = 0; j < gamma; ++j)
            acc = fmaf(-E[j], U[(size_t)(b0 + j) * cols + f], acc);
          T[f] = acc;
        }
      }
      /* the residual chain of the original row after this level's codes */
      for (int G = 0; G < ng; ++G) {
        const size_t gi = (size_t)n * ng + G;
        const int c0 = G * group;
        if (lev == 0) {
          for (int k = 0; k < group; ++k) R[c0 + k] = w[c0 + k] - what[c0 + k];
        } else {
          const float sb = oracle_f16_to_f32(scales[(size_t)lev * rows * ng + gi]);
          const uint8_t* sg = signs + (size_t)(lev - 1) * rows * cols + (size_t)n * cols + c0;
          for (int k = 0; k < group; ++k)
            R[c0 + k] = sg[k] ? (R[c0 + k] - sb) : (R[c0 + k] + sb);
        }
      }
    }
  }
  free(T); free(R); free(what); free(D); free(E);
  return 0;
}

/* W^_b = (Q_b1 - z) s_b1 + sum_{levels 1..b-b1} s_l * sigma_l  (exact). */
int oracle_mwq_dequant(int rows, int cols, int group, int b_min, int b_max,
                       int b, const uint8_t* q1, const uint8_t* zeros,
                       const uint16_t* scales, const uint8_t* signs,
                       double* What) {
  if (rows <= 0 || cols <= 0 || group <= 0 || cols % group != 0 ||
      !check_ladder(b_min, b_max) || b < b_min || b > b_max || !What)
    return -1;
  const int ng = cols / group;
  for (int n = 0; n < rows; ++n) {
    for (int k = 0; k < cols; ++k) {
      const size_t gi = (size_t)n * ng + k / group;
      const size_t wi = (size_t)n * cols + k;
      double v = (double)((int)q1[wi] - (int)zeros[gi]) *
                 (double)oracle_f16_to_f32(scales[gi]);
      for (int lev = 1; lev <= b - b_min; ++lev) {
        const double s =
            (double)oracle_f16_to_f32(scales[(size_t)lev * rows * ng + gi]);
        const int pos = signs[(size_t)(lev - 1) * rows * cols + wi];
        v = v + (pos ? s : -s);
      }
      What[wi] = v;
    }
  }
  return 0;
}

/* ---- canonical tiled bit-plane layout ---------------------------------- */

int oracle_mwq_pack(int rows, int cols, int group, int b_min, int b_max,
                    const uint8_t* q1, const uint8_t* zeros,
                    const uint16_t* scales, const uint8_t* signs,
                    uint32_t* planes, uint16_t* scales_out,
                    uint8_t* zeros_out) {
  if ((group != 64 && group != 128) || !check_ladder(b_min, b_max) ||
      rows <= 0 || cols <= 0 || cols % group != 0)
    return -1;
  const int BR = 2048 / group;
  if (rows % BR != 0) return -1;
  const int KB = cols / group, P = b_max, levels = b_max - b_min + 1;
  const int ng = KB;
  const size_t nwords = (size_t)rows * cols / 32 * P;
  memset(planes, 0, nwords * 4);

  for (int n = 0; n < rows; ++n) {
    const int rb = n / BR, i = n % BR;
    for (int k = 0; k < cols; ++k) {
      const int kb = k / group, kk = k % group;
      const int sub = kk / 32, bit = kk % 32;
      const int w = sub * BR + i;
      const size_t blk = (size_t)rb * KB + kb;
      const size_t wi = (size_t)n * cols + k;
      for (int p = 0; p < P; ++p) {
        int v;
        if (p < b_min)
          v = (q1[wi] >> p) & 1;
        else
          v = signs[(size_t)(p - b_min) * rows * cols + wi] & 1;
        if (v) planes[(blk * P + p) * 64 + w] |= (uint32_t)1u << bit;
      }
    }
    for (int G = 0; G < ng; ++G) {
      const size_t blk = (size_t)rb * KB + G;
      const size_t gi = (size_t)n * ng + G;
      zeros_out[blk * BR + i] = zeros[gi];
      for (int lev = 0; lev < levels; ++lev)
        scales_out[(blk * levels + lev) * BR + i] =
            scales[(size_t)lev * rows * ng + gi];
    }
  }
  return 0;
}

/* ---- dual routing ------------------------------------------------------ */

int oracle_gate_logits(const float* x, int T, int d, const float* Wg,
                       const float* bias, int E, double* logits) {
  if (!x || !Wg || !logits || T < 0 || d <= 0 || E <= 0) return -1;
  for (int t = 0; t < T; ++t)
    for (int e = 0; e < E; ++e) {
      double acc = 0.0;
      for (int c = 0; c < d; ++c)
        acc += (double)x[(size_t)t * d + c] * (double)Wg[(size_t)e * d + c];
      if (bias) acc += (double)bias[e];
      logits[(size_t)t * E + e] = acc;
    }
  return 0;
}

int oracle_route_from_logits(const double* logits, int T, int E, int k,
                             const int* token_req, const uint8_t* bit_table,
                             int R, int b_min, int b_max, int* topk_idx,
                             double* topk_w, uint8_t* topk_bits, int* hist,
                             int* offsets, int* perm, int* slot_of,
                             uint8_t* maxbit) {
  if (T < 0 || E <= 0 || k <= 0 || k > E || R <= 0 ||
      !check_ladder(b_min, b_max))
    return -1;
  const int L = b_max - b_min + 1;
  int bad = 0;
  char* taken = (char*)malloc((size_t)E);
  if (!taken) return -1;

  for (int t = 0; t < T; ++t) {
    const double* l = logits + (size_t)t * E;
    memset(taken, 0, (size_t)E);
    /* the first k entries of a stable sort by (logit desc, index asc) */
    for (int i = 0; i < k; ++i) {
      int best = -1;
      for (int e = 0; e < E; ++e) {
        if (taken[e]) continue;
        if (best < 0 || l[e] > l[best]) best = e;
      }
      taken[best] = 1;
      topk_idx[t * k + i] = best;
    }
    /* softmax over the selected logits (Mixtral-style renormalised gate) */
    const double lmax = l[topk_idx[t * k]];
    double den = 0.0;
    for (int i = 0; i < k; ++i) den += exp(l[topk_idx[t * k + i]] - lmax);
    for (int i = 0; i < k; ++i)
      topk_w[t * k + i] = exp(l[topk_idx[t * k + i]] - lmax) / den;
    /* bit-width of each activated expert: per (request, expert) table */
    const int r = token_req ? token_req[t] : 0;
    for (int i = 0; i < k; ++i) {
      int b = b_min;
      if (r < 0 || r >= R) {
        bad = 1;
      } else {
        b = bit_table[(size_t)r * E + topk_idx[t * k + i]];
        if (b < b_min || b > b_max) bad = 1;
      }
      topk_bits[t * k + i] = (uint8_t)b;
    }
  }
  free(taken);
  if (bad) return -2;

  /* selection counts per (expert, bit-width), exclusive scan, stable sort */
  for (int j = 0; j < E * L; ++j) hist[j] = 0;
  for (int s = 0; s < T * k; ++s)
    hist[topk_idx[s] * L + (topk_bits[s] - b_min)] += 1;
  offsets[0] = 0;
  for (int j = 0; j < E * L; ++j) offsets[j + 1] = offsets[j] + hist[j];
  int* fill = (int*)calloc((size_t)E * L, sizeof(int));
  if (!fill) return -1;
  for (int s = 0; s < T * k; ++s) {
    const int key = topk_idx[s] * L + (topk_bits[s] - b_min);
    const int pos = offsets[key] + fill[key]++;
    perm[pos] = s;
    slot_of[s] = pos;
  }
  free(fill);
  for (int e = 0; e < E; ++e) {
    int mb = 0;
    for (int j = 0; j < L; ++j)
      if (hist[e * L + j] > 0) mb = b_min + j;
    maxbit[e] = (uint8_t)mb;
  }
  return 0;
}

/* ---- expert FFN and combine -------------------------------------------- */

static double dequant_elem(int rows, int cols, int group, int b_min, int b,
                           const uint8_t* q1, const uint8_t* zeros,
                           const uint16_t* scales, const uint8_t* signs,
                           int n, int c) {
  const int ng = cols / group;
  const size_t gi = (size_t)n * ng + c / group;
  const size_t wi = (size_t)n * cols + c;
  double v = (double)((int)q1[wi] - (int)zeros[gi]) *
             (double)oracle_f16_to_f32(scales[gi]);
  for (int lev = 1; lev <= b - b_min; ++lev) {
    const double s =
        (double)oracle_f16_to_f32(scales[(size_t)lev * rows * ng + gi]);
    v = v + (signs[(size_t)(lev - 1) * rows * cols + wi] ? s : -s);
  }
  return v;
}

static double silu(double a) { return a / (1.0 + exp(-a)); }

int oracle_expert_ffn(int d, int f, int d_out, int group13, int group2, int b_min,
                      int b_max, int b,
                      const uint8_t* q1_13, const uint8_t* zeros_13,
                      const uint16_t* scales_13, const uint8_t* signs_13,
                      const uint8_t* q1_2, const uint8_t* zeros_2,
                      const uint16_t* scales_2, const uint8_t* signs_2,
                      const double* x, int n, double* y) {
  if (d <= 0 || f <= 0 || d_out <= 0 || n < 0 || !check_ladder(b_min, b_max) ||
      b < b_min || b > b_max || d % group13 != 0 || f % group2 != 0)
    return -1;
  double* h = (double*)malloc(sizeof(double) * (size_t)f * (n > 0 ? n : 1));
  double* wa = (double*)malloc(sizeof(double) * (size_t)d);
  double* wc = (double*)malloc(sizeof(double) * (size_t)d);
  double* w2 = (double*)malloc(sizeof(double) * (size_t)f);
  if (!h || !wa || !wc || !w2) {
    free(h); free(wa); free(wc); free(w2);
    return -1;
  }
  /* a = W1_b x and c = W3_b x, one weight row at a time */
  for (int r = 0; r < f; ++r) {
    for (int c = 0; c < d; ++c) {
      wa[c] = dequant_elem(2 * f, d, group13, b_min, b, q1_13, zeros_13,
                           scales_13, signs_13, r, c);
      wc[c] = dequant_elem(2 * f, d, group13, b_min, b, q1_13, zeros_13,
                           scales_13, signs_13, f + r, c);
    }
    for (int j = 0; j < n; ++j) {
      const double* xj = x + (size_t)j * d;
      double a = 0.0, cc = 0.0;
      for (int c = 0; c < d; ++c) a += wa[c] * xj[c];
      for (int c = 0; c < d; ++c) cc += wc[c] * xj[c];
      h[(size_t)j * f + r] = silu(a) * cc;
    }
  }
  /* y = W2_b h */
  for (int r = 0; r < d_out; ++r) {
    for (int c = 0; c < f; ++c)
      w2[c] = dequant_elem(d_out, f, group2, b_min, b, q1_2, zeros_2, scales_2,
                           signs_2, r, c);
    for (int j = 0; j < n; ++j) {
      const double* hj = h + (size_t)j * f;
      double acc = 0.0;
      for (int c = 0; c < f; ++c) acc += w2[c] * hj[c];
      y[(size_t)j * d_out + r] = acc;
    }
  }
  free(h); free(wa); free(wc); free(w2);
  (void)b_max;
  return 0;
}

/* ---- decoder stack: normalisation before each MoE layer -------------- */

int oracle_rmsnorm(int T, int d, double eps, const double* x, double* h) {
  if (T < 0 || d <= 0 || !(eps >= 0.0)) return -1;
  for (int t = 0; t < T; ++t) {
    const double* row = x + (size_t)t * d;
    double ss = 0.0;
    for (int c = 0; c < d; ++c) ss += row[c] * row[c];
    const double inv = 1.0 / sqrt(ss / (double)d + eps);
    for (int c = 0; c < d; ++c) h[(size_t)t * d + c] = row[c] * inv;
  }
  return 0;
}

int oracle_combine(int T, int k, int d, const double* topk_w,
                   const double* y_slot, double* out) {
  if (T < 0 || k <= 0 || d <= 0) return -1;
  for (int t = 0; t < T; ++t)
    for (int c = 0; c < d; ++c) {
      double acc = 0.0;
      for (int i = 0; i < k; ++i)
        acc += topk_w[t * k + i] * y_slot[((size_t)t * k + i) * d + c];
      out[(size_t)t * d + c] = acc;
    }
  return 0;
}
