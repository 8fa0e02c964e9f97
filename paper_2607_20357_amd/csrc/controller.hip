// LLM-side compute controller (Sec. 3.2) and the row moves of the controlled
// prefill.
//
//   * ctrl_stats_kernel: per sample, the threshold count (z > 0) and the soft
//     survival rate kappa = sum_i sigma(z_i) / N in float64 (Eq. (7));
//   * pe_kernel: the sinusoidal encoding of a scalar (the budget b, or each
//     sample's kappa), computed in float64 and stored as float32;
//   * linear_kernel: y = act(W x + bias) (+ a residual row), the small
//     matrix-vector products of MLP_LLM, MLP_kappa and the gating head.  One
//     wave per output row streams that row of W once (16-byte loads, a wave
//     reads 1 KiB per step) for up to 8 input vectors; the lane sums are
//     reduced in a fixed order, so results do not depend on the launch;
//   * budget_rows_kernel: writes the budget token into the last row of every
//     sample's packed sequence;
//   * compact_rows_kernel: removes the rows of the visual tokens that the
//     budget projection discards at the prefix boundary, keeping the order of
//     the others.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;
constexpr int LIN_NV = 8;   // input vectors per pass of the linear kernel

__global__ __launch_bounds__(NT) void ctrl_stats_kernel(const float* z, int N, int32_t* counts,
                                                        double* kappa) {
  __shared__ int s_cnt[NT / 64];
  __shared__ double s_sum[NT / 64];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* zb = z + (size_t)b * N;
  int n = 0;
  double s = 0.0;
  for (int i = tid; i < N; i += NT) {
    const float v = zb[i];
    n += v > 0.0f ? 1 : 0;
    if (v == v) {   // sigma(NaN) counts as 0
      const double x = (double)v;
      if (x >= 0.0) {
        s += 1.0 / (1.0 + exp(-x));
      } else {
        const double e = exp(x);
        s += e / (1.0 + e);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    n += __shfl_xor(n, o, 64);
    s += __shfl_xor(s, o, 64);
  }
  if ((tid & 63) == 0) {
    s_cnt[tid >> 6] = n;
    s_sum[tid >> 6] = s;
  }
  __syncthreads();
  if (tid == 0) {
    int tn = 0;
    double ts = 0.0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) { tn += s_cnt[i]; ts += s_sum[i]; }
    counts[b] = tn;
    kappa[b] = N > 0 ? ts / (double)N : 0.0;
  }
}

// grid (ceil(E/2 / NT), nvec): out[r][2i] = sin(x w_i), out[r][2i+1] = cos(x w_i),
// x = (xs ? xs[r] : x0) * scale, w_i = base^(-2i/E).
__global__ __launch_bounds__(NT) void pe_kernel(const double* xs, double x0, int E, double scale,
                                                double base, float* out) {
  const int r = blockIdx.y;
  const int i = blockIdx.x * NT + threadIdx.x;
  if (2 * i >= E) return;
  const double x = (xs ? xs[r] : x0) * scale;
  const double w = pow(base, -2.0 * (double)i / (double)E);
  out[(size_t)r * E + 2 * i] = (float)sin(x * w);
  out[(size_t)r * E + 2 * i + 1] = (float)cos(x * w);
}

template <bool BF16>
__device__ __forceinline__ void load_w8(const void* W, size_t off, float (&w)[8]) {
  if constexpr (BF16) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(W) + off);
    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      w[2 * e] = bf16_bits_to_f32(u[e] & 0xffffu);
      w[2 * e + 1] = bf16_bits_to_f32(u[e] >> 16);
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(W) + off);
    const float4 a = p[0], c = p[1];
    w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
    w[4] = c.x; w[5] = c.y; w[6] = c.z; w[7] = c.w;
  }
}

template <bool BF16>
__device__ __forceinline__ float load_w1(const void* W, size_t off) {
  if constexpr (BF16) return bf16_bits_to_f32(static_cast<const uint16_t*>(W)[off]);
  else return static_cast<const float*>(W)[off];
}

// One wave per output row o (4 rows per workgroup).  Each lane takes 8
// consecutive inputs per 512-input step and issues the weight loads of LIN_U
// steps before using them, so every wave keeps LIN_U 1 KiB row pieces in
// flight.
constexpr int LIN_U = 4;

template <bool BF16>
__global__ __launch_bounds__(NT) void linear_kernel(CtrlLinearArgs a) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
  if (o >= a.out) return;
  const size_t wrow = (size_t)o * a.in;
  for (int r0 = 0; r0 < a.nvec; r0 += LIN_NV) {
    const int nv = min(LIN_NV, a.nvec - r0);
    float acc[LIN_NV];
#pragma unroll
    for (int r = 0; r < LIN_NV; ++r) acc[r] = 0.f;
    for (int k0 = lane * 8; k0 < a.in; k0 += 64 * 8 * LIN_U) {
      float w[LIN_U][8];
#pragma unroll
      for (int u = 0; u < LIN_U; ++u) {
        const int k = k0 + u * 64 * 8;
        if (k < a.in) load_w8<BF16>(a.W, wrow + k, w[u]);
      }
#pragma unroll
      for (int r = 0; r < LIN_NV; ++r) {
        if (r < nv) {
          const float* xr = a.x + (size_t)(r0 + r) * a.ldx;
#pragma unroll
          for (int u = 0; u < LIN_U; ++u) {
            const int k = k0 + u * 64 * 8;
            if (k < a.in) {
              const float4* xp = reinterpret_cast<const float4*>(xr + k);
              const float4 x0 = xp[0], x1 = xp[1];
              acc[r] += w[u][0] * x0.x + w[u][1] * x0.y + w[u][2] * x0.z + w[u][3] * x0.w +
                        w[u][4] * x1.x + w[u][5] * x1.y + w[u][6] * x1.z + w[u][7] * x1.w;
            }
          }
        }
      }
    }
    const float bias = a.bias ? load_w1<BF16>(a.bias, o) : 0.f;
#pragma unroll
    for (int r = 0; r < LIN_NV; ++r) {
      if (r < nv) {
        float v = warp_sum(acc[r]) + bias;
        if (a.act == CTRL_ACT_GELU) v = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
        if (lane == 0) {
          const int vec = r0 + r;
          if (a.add) {
            const int64_t row = a.add_cu ? (int64_t)a.add_cu[vec + 1] - 1 : vec;
            v += a.add[row * a.ldadd + o];
          }
          a.y[(size_t)vec * a.ldy + o] = v;
        }
      }
    }
  }
}

// grid B: resid[cu[b+1]-1][:] = eb[:]
__global__ __launch_bounds__(NT) void budget_rows_kernel(const float* eb, const int32_t* cu, int D,
                                                         float* resid) {
  const int b = blockIdx.x;
  float* dst = resid + ((size_t)cu[b + 1] - 1) * D;
  for (int c = threadIdx.x; c < D / 4; c += NT)
    reinterpret_cast<float4*>(dst)[c] = reinterpret_cast<const float4*>(eb)[c];
}

// grid = rows of the new packing.  Row i of sample b is its i-th kept visual
// token (found among the old kept list, ascending, by binary search) or, past
// the kept tokens, the text / budget row at the same distance from the end of
// the visual block.
__global__ __launch_bounds__(NT) void compact_rows_kernel(CompactArgs a) {
  const int r = blockIdx.x;
  int lo = 0, hi = a.B - 1;   // sample b with new_cu[b] <= r < new_cu[b+1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.new_cu[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int b = lo, i = r - a.new_cu[b];
  const int k2 = a.new_keep[b], k1 = a.old_keep[b];
  int64_t src;
  if (i < k2) {
    const int idx = a.new_kidx[(size_t)b * a.N + i];
    const int32_t* old = a.old_kidx + (size_t)b * a.N;
    int l = 0, h = k1 - 1;   // first position with old[pos] >= idx
    while (l < h) {
      const int m = (l + h) >> 1;
      if (old[m] < idx) l = m + 1; else h = m;
    }
    src = (int64_t)a.old_cu[b] + l;
  } else {
    src = (int64_t)a.old_cu[b] + k1 + (i - k2);
  }
  const float4* s = reinterpret_cast<const float4*>(a.src + src * a.D);
  float4* d = reinterpret_cast<float4*>(a.dst + (int64_t)r * a.D);
  for (int c = threadIdx.x; c < a.D / 4; c += NT) d[c] = s[c];
}

}  // namespace

hipError_t launch_ctrl_stats(const float* z, int32_t B, int32_t N, int32_t* counts, double* kappa,
                             hipStream_t st) {
  if (B <= 0) return hipSuccess;
  ctrl_stats_kernel<<<B, NT, 0, st>>>(z, N, counts, kappa);
  return hipGetLastError();
}

hipError_t launch_pe(const double* xs, double x0, int32_t nvec, int32_t E, double scale,
                     double base, float* out, hipStream_t st) {
  if (nvec <= 0 || E <= 0) return hipSuccess;
  const dim3 grid((unsigned)((E / 2 + NT - 1) / NT), (unsigned)nvec);
  pe_kernel<<<grid, NT, 0, st>>>(xs, x0, E, scale, base, out);
  return hipGetLastError();
}

hipError_t launch_ctrl_linear(const CtrlLinearArgs& a, bool bf16, hipStream_t st) {
  if (a.out <= 0 || a.nvec <= 0) return hipSuccess;
  if (a.in % 8) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((a.out + NT / 64 - 1) / (NT / 64));
  if (bf16) linear_kernel<true><<<grid, NT, 0, st>>>(a);
  else linear_kernel<false><<<grid, NT, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_budget_rows(const float* eb, const int32_t* cu, int32_t B, int32_t D,
                              float* resid, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  if (D % 4) return hipErrorInvalidValue;
  budget_rows_kernel<<<B, NT, 0, st>>>(eb, cu, D, resid);
  return hipGetLastError();
}

hipError_t launch_compact_rows(const CompactArgs& a, int32_t rows, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (a.D % 4) return hipErrorInvalidValue;
  compact_rows_kernel<<<rows, NT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace svl
