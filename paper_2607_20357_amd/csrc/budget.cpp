// Budget projection (Sec. 3.3 "Inference"): host arithmetic.
//
// Cost of one sample with S = n_text + s kept tokens (Eq. (8)):
//   C(s) = sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2] + 2 D V S,
// alpha_l = a_l / A with a_l the active query heads of an executed layer (0
// for a skipped one).  Everything is kept exact: A * C(s) is an integer
// (sum of a_l times the layer term, plus A times the LM-head term), and the
// float budget b is m * 2^q with an integer m, so C(s) <= b * C_full is
// decided on 128-bit integers.
#include "budget.h"

#include <algorithm>
#include <cmath>
#include <tuple>
#include <vector>

namespace svl {
namespace {

using i128 = __int128;

int bitlen(i128 x) {
  int n = 0;
  while (x > 0) { x >>= 1; ++n; }
  return n;
}

// A * C at sequence length S, with sum_a = sum over executed layers of a_l.
i128 cost_times_heads(const svl_config& c, int64_t S, int64_t sum_a, int64_t vocab) {
  const i128 D = c.d_model, F = c.d_ffn, A = c.n_heads;
  const i128 layer = (8 * D * D + 6 * D * F) * (i128)S + 4 * D * (i128)S * S;
  return (i128)sum_a * layer + A * 2 * D * (i128)vocab * S;
}

// x <= b * y for integers x, y >= 0 and a float 0 < b < 1, exactly.
bool fits(i128 x, float b, i128 y) {
  if (x == 0) return true;
  int e = 0;
  const float m = std::frexp(b, &e);                 // b = m 2^e, m in [0.5, 1)
  const int64_t mi = (int64_t)std::ldexp(m, 24);     // b = mi 2^(e - 24), mi < 2^24
  const int sh = 24 - e;                              // b < 1: e <= 0, so sh >= 24
  const i128 r = (i128)mi * y;                        // compare x 2^sh with r
  const int bx = bitlen(x), br = bitlen(r);
  if (bx + sh > br) return false;                     // x 2^sh >= 2^(bx-1+sh) >= 2^br > r
  return (x << sh) <= r;                              // fits: bx + sh <= br <= 126
}

int64_t active_heads(const svl_config& c, const uint8_t* layer_on, const uint8_t* head_on) {
  int64_t n = 0;
  for (int32_t l = 0; l < c.n_layers; ++l)
    if (layer_on[l])
      for (int32_t h = 0; h < c.n_heads; ++h) n += head_on[(int64_t)l * c.n_heads + h] != 0;
  return n;
}

// Largest s in [0, n_pos] with C(s) <= b C_full (C grows with s), or -1.
int32_t max_tokens(const svl_config& c, int32_t n_text, int32_t n_pos, int64_t sum_a,
                   int64_t vocab, float b, i128 full) {
  if (!fits(cost_times_heads(c, n_text, sum_a, vocab), b, full)) return -1;
  int32_t lo = 0, hi = n_pos;                          // C(lo) fits
  while (lo < hi) {
    const int32_t mid = lo + (hi - lo + 1) / 2;
    if (fits(cost_times_heads(c, (int64_t)n_text + mid, sum_a, vocab), b, full)) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

}  // namespace

int32_t project_budget_sample(const svl_config& c, int32_t n_vision, int32_t n_text,
                              int32_t n_pos, float budget, int64_t vocab, int32_t prefix,
                              uint8_t* layer_on, uint8_t* head_on, uint8_t* ffn_on,
                              const float* gate_logits, int32_t units) {
  if (budget >= 1.0f) return n_pos;
  const int64_t L = c.n_layers, A = c.n_heads, G = units, hg = A / G;
  const i128 full = cost_times_heads(c, (int64_t)n_text + n_vision, L * A, vocab);
  int64_t sum_a = active_heads(c, layer_on, head_on);
  const int32_t s = max_tokens(c, n_text, n_pos, sum_a, vocab, budget, full);
  if (s >= 0) return s;
  // Even no visual token fits: switch off whole head groups of layers at or
  // after the prefix, lowest gate logit first (ties: later layer, higher group).
  // With one unit per layer (layer controller) a unit is the whole layer.
  std::vector<std::tuple<float, int64_t, int64_t>> order;   // (logit, -layer, -group)
  for (int64_t l = prefix; l < L; ++l) {
    if (!layer_on[l]) continue;
    for (int64_t j = 0; j < G; ++j) {
      bool any = false;
      for (int64_t h = j * hg; h < (j + 1) * hg; ++h) any = any || head_on[l * A + h];
      if (any) order.emplace_back(gate_logits ? gate_logits[l * G + j] : 0.0f, -l, -j);
    }
  }
  std::sort(order.begin(), order.end());
  for (const auto& u : order) {
    const int64_t l = -std::get<1>(u), j = -std::get<2>(u);
    for (int64_t h = j * hg; h < (j + 1) * hg; ++h) head_on[l * A + h] = 0;
    if (ffn_on) {
      if (G == 1) { for (int64_t q = 0; q < c.n_groups; ++q) ffn_on[l * c.n_groups + q] = 0; }
      else ffn_on[l * G + j] = 0;
    }
    bool any = false;
    for (int64_t h = 0; h < A; ++h) any = any || head_on[l * A + h];
    if (!any) layer_on[l] = 0;
    sum_a = active_heads(c, layer_on, head_on);
    const int32_t t = max_tokens(c, n_text, n_pos, sum_a, vocab, budget, full);
    if (t >= 0) return t;
  }
  return 0;
}

}  // namespace svl
