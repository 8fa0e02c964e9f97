// Training-time budget term (Sec. 3.1 Eq. (6), Sec. 3.3 Eq. (8)-(10)): the
// controllers' straight-through decisions, the differentiable cost ratio and
// the asymmetric budget loss with its gradient with respect to the token and
// gate logits.  One workgroup per sample; sums in float64 with a fixed
// reduction order, so results do not depend on the launch.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;

__device__ __forceinline__ double sigmoid_d(double x) {
  if (x >= 0.0) return 1.0 / (1.0 + exp(-x));
  const double e = exp(x);
  return e / (1.0 + e);
}

__device__ __forceinline__ double block_sum_d(double v, double* s_red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();   // s_red free (an earlier reduction's readers are done)
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r += s_red[i];
  return r;
}

__global__ __launch_bounds__(NT) void budget_loss_kernel(BudgetLossArgs a) {
  __shared__ double s_red[NT / 64];
  __shared__ double s_coef[2];   // dL/dr dr/dS;  dL/dr dr/dalpha / (U tau_comp)
  const int b = blockIdx.x, tid = threadIdx.x;
  const int nl = (a.L - a.P) * a.U;
  const float* z = a.z + (size_t)b * a.N;
  const float* xt = a.xi_tok ? a.xi_tok + (size_t)b * a.N : nullptr;
  const float* g = a.gl + (size_t)b * nl;
  const float* xg = a.xi_gate ? a.xi_gate + (size_t)b * nl : nullptr;

  // token decisions (z + xi > 0) and the soft count sum sigma(z)
  double soft = 0.0;
  for (int i = tid; i < a.N; i += NT) {
    const double v = (double)z[i] + (xt ? (double)xt[i] : 0.0);
    a.tok_mask[(size_t)b * a.N + i] = v > 0.0 ? 1 : 0;
    soft += sigmoid_d((double)z[i]);
  }
  soft = block_sum_d(soft, s_red);

  // unit decisions and the layer activities alpha_l = (units on) / U
  double act = 0.0;
  for (int l = tid; l < a.L - a.P; l += NT) {
    int on = 0;
    for (int j = 0; j < a.U; ++j) {
      const int u = l * a.U + j;
      const double v = (double)g[u] + (xg ? (double)xg[u] : 0.0);
      const int m = v > 0.0 ? 1 : 0;
      a.unit_mask[(size_t)b * nl + u] = (uint8_t)m;
      on += m;
    }
    act += (double)on / (double)a.U;
  }
  act = block_sum_d(act, s_red) + (double)a.P;   // prefix layers at alpha = 1

  if (tid == 0) {
    const double S = (double)a.T + soft;
    const double per_layer = a.c1 * S + a.c2 * S * S;
    const double cost = act * per_layer + a.lm * S;
    const double r = cost / a.full;
    const double over = fmax(0.0, r - a.budget);
    const double under = fmax(0.0, (a.budget - a.margin) - r);
    const double loss = a.lam * (a.w_over * over * over + a.w_under * under);
    const double dldr = a.lam * (2.0 * a.w_over * over - (under > 0.0 ? a.w_under : 0.0));
    const double drds = (act * (a.c1 + 2.0 * a.c2 * S) + a.lm) / a.full;
    s_coef[0] = dldr * drds;
    s_coef[1] = dldr * (per_layer / a.full) / ((double)a.U * a.tau_comp);
    a.ratio[b] = (float)r;
    a.loss[b] = (float)loss;
  }
  __syncthreads();
  const double cz = s_coef[0], cg = s_coef[1];
  for (int i = tid; i < a.N; i += NT) {
    const double s = sigmoid_d((double)z[i]);
    a.grad_z[(size_t)b * a.N + i] = (float)(cz * s * (1.0 - s));
  }
  for (int u = tid; u < nl; u += NT) {
    const double y = sigmoid_d(((double)g[u] + (xg ? (double)xg[u] : 0.0)) / a.tau_comp);
    a.grad_gate[(size_t)b * nl + u] = (float)(cg * y * (1.0 - y));
  }
}

}  // namespace

hipError_t launch_budget_loss(const BudgetLossArgs& a, int32_t B, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  budget_loss_kernel<<<B, NT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace svl
