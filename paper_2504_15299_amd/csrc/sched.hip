// Host-side planning of the bit-width-aware I/O-compute pipeline (Sec. 3.4)
// for weights that are streamed into device memory instead of held there:
// the Hottest-Expert-Bit-First (HEBF) order of the (expert, bit-width) units
// of one layer (Sec. 3.4.3), and the memory-budget scheduler of Algorithm 2
// (Sec. 3.4.1) that decides which levels of earlier layers to release when
// the next layer does not fit.  Plain host code, no allocation.
#include "internal.h"

namespace d2moe {

// HEBF: a queue per expert of its requested bit-widths in ascending order;
// repeatedly the head with the largest count B_{j,k} (ties: lower expert)
// joins the I/O queue.  Each unit's load is the expert's nested delta from
// the width already present to the unit's width.  Returns the unit count.
int hebf_order(const int32_t* hist, int E, int b_min, int b_max, const uint8_t* resident,
               d2moe_unit* units) {
  const int L = b_max - b_min + 1;
  int head[64], have[64];
  for (int j = 0; j < E; ++j) {
    head[j] = 0;
    while (head[j] < L && hist[j * L + head[j]] <= 0) ++head[j];
    have[j] = resident ? resident[j] : 0;
  }
  int n = 0;
  for (;;) {
    int best = -1, bc = 0;
    for (int j = 0; j < E; ++j) {
      if (head[j] >= L) continue;
      const int c = hist[j * L + head[j]];
      if (best < 0 || c > bc) {
        best = j;
        bc = c;
      }
    }
    if (best < 0) break;
    const int bits = b_min + head[best];
    d2moe_unit& u = units[n++];
    u.expert = best;
    u.bits = bits;
    u.load_from = have[best];
    u.load_to = have[best] > bits ? have[best] : bits;
    u.count = bc;
    have[best] = u.load_to;
    ++head[best];
    while (head[best] < L && hist[best * L + head[best]] <= 0) ++head[best];
  }
  return n;
}

// Algorithm 2 over one pass of the layers (levels: 0 = base planes with
// their scale and zero points, l >= 1 = one residual plane with its
// scales).  For each layer, when the levels it still needs do not fit the
// free budget, levels of earlier layers are released, the previous layer
// first, its highest level first (one level of every expert of that layer at
// a time, experts ascending), the base level last, until they fit; then the
// layer's levels are loaded.  Returns the number of actions, or -(number
// needed) - 1 if max_actions is too small (actions past it are not written).
int budget_plan(const uint8_t* want, int n_layers, int E, const int64_t* level_bytes, int K,
                int64_t budget, uint8_t* res, d2moe_budget_action* actions, int max_actions) {
  int64_t used = 0;
  for (int j = 0; j < n_layers; ++j)
    for (int e = 0; e < E; ++e)
      for (int l = 0; l < res[j * E + e]; ++l) used += level_bytes[l];
  int64_t free_b = budget - used;
  int n = 0;
  auto emit = [&](int act, int j, int e, int l) {
    if (n < max_actions) actions[n] = d2moe_budget_action{act, j, e, l};
    ++n;
  };
  for (int j = 0; j < n_layers; ++j) {
    int64_t need = 0;
    for (int e = 0; e < E; ++e)
      for (int l = res[j * E + e]; l < want[j * E + e]; ++l) need += level_bytes[l];
    for (int jj = j - 1; jj >= 0 && need > free_b; --jj) {
      for (int l = K - 1; l >= 0 && need > free_b; --l) {
        for (int e = 0; e < E; ++e) {
          if (res[jj * E + e] == l + 1) {
            emit(0, jj, e, l);
            res[jj * E + e] = (uint8_t)l;
            free_b += level_bytes[l];
          }
        }
      }
    }
    for (int e = 0; e < E; ++e) {
      for (int l = res[j * E + e]; l < want[j * E + e]; ++l) {
        emit(1, j, e, l);
        free_b -= level_bytes[l];
      }
      if (want[j * E + e] > res[j * E + e]) res[j * E + e] = want[j * E + e];
    }
  }
  return n <= max_actions ? n : -n - 1;
}

}  // namespace d2moe
