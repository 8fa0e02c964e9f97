// RMSNorm of the residual rows that run a sub-block, the RoPE (cos, sin)
// table, and a fill kernel.
//
// RMSNorm: one workgroup per row, float32 statistics over the float32
// residual, output y = x * rsqrt(mean(x^2) + eps) * gain in the activation
// type (fp16 or bf16 for the MFMA path, float32 for the float32 path); the
// gain is stored in the weight dtype.  Only rows of samples that execute the
// sub-block are listed, so skipped samples are neither read nor written.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;

// OUT: 0 float32 (float32 gain), 1 bf16, 2 fp16 (bf16 gain)
template <int OUT>
__global__ __launch_bounds__(NT) void rmsnorm_kernel(NormArgs a) {
  __shared__ float s_part[NT / 64];
  const int r = blockIdx.x;
  int lo = 0, hi = a.nsegs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].prefix <= r) lo = mid; else hi = mid - 1;
  }
  const Seg sg = a.segs[lo];
  const size_t row = (size_t)sg.row0 + (r - sg.prefix);
  const int D = a.D, tid = threadIdx.x;
  const float4* x = reinterpret_cast<const float4*>(a.x + row * D);
  float ss = 0.f;
  for (int c = tid; c < D / 4; c += NT) {
    const float4 v = x[c];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = warp_sum(ss);
  if ((tid & 63) == 0) s_part[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) tot += s_part[i];
  const float inv = rsqrtf(tot / (float)D + a.eps);
  if constexpr (OUT != 0) {
    const uint2* gain = reinterpret_cast<const uint2*>(a.gain);
    uint2* out = reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + row * D);
    for (int c = tid; c < D / 4; c += NT) {
      const float4 v = x[c];
      const uint2 gw = gain[c];
      const float g0 = bf16_bits_to_f32(gw.x & 0xffffu), g1 = bf16_bits_to_f32(gw.x >> 16);
      const float g2 = bf16_bits_to_f32(gw.y & 0xffffu), g3 = bf16_bits_to_f32(gw.y >> 16);
      out[c] = make_uint2(pack_act2<OUT == 2>(v.x * inv * g0, v.y * inv * g1),
                          pack_act2<OUT == 2>(v.z * inv * g2, v.w * inv * g3));
    }
  } else {
    const float4* gain = reinterpret_cast<const float4*>(a.gain);
    float4* out = reinterpret_cast<float4*>(static_cast<float*>(a.out) + row * D);
    for (int c = tid; c < D / 4; c += NT) {
      const float4 v = x[c], g = gain[c];
      out[c] = make_float4(v.x * inv * g.x, v.y * inv * g.y, v.z * inv * g.z, v.w * inv * g.w);
    }
  }
}

// table[p][r] = (cos, sin)(p * theta^(-2r/d)), evaluated in double.
__global__ void rope_table_kernel(float2* table, int max_pos, int half, double theta) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= max_pos * half) return;
  const int p = idx / half, r = idx % half;
  const double w = pow(theta, -2.0 * (double)r / (double)(2 * half));
  double sn, cs;
  sincos((double)p * w, &sn, &cs);
  table[idx] = make_float2((float)cs, (float)sn);
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

hipError_t launch_rmsnorm(const NormArgs& a, int32_t out_kind, hipStream_t st) {
  if (a.nrows <= 0) return hipSuccess;
  if (out_kind == 2) rmsnorm_kernel<2><<<a.nrows, NT, 0, st>>>(a);
  else if (out_kind == 1) rmsnorm_kernel<1><<<a.nrows, NT, 0, st>>>(a);
  else rmsnorm_kernel<0><<<a.nrows, NT, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* table, int32_t max_pos, int32_t head_dim, float theta,
                             hipStream_t st) {
  const int half = head_dim / 2;
  const int64_t n = (int64_t)max_pos * half;
  if (n <= 0) return hipSuccess;
  rope_table_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(table, max_pos, half,
                                                                   (double)theta);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t value, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  fill_i32_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(p, value, n);
  return hipGetLastError();
}

}  // namespace svl
