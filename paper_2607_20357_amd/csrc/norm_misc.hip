// Residual finish + RMSNorm, the RoPE (cos, sin) table, and a fill kernel.
//
// Residual finish + RMSNorm: one workgroup per listed row.  Rows flagged
// NORM_ADD_PARTIALS first receive the pending split-K partial slices of the
// previous output / down projection, added in slice order (a fixed order:
// the result does not depend on scheduling), and are written back.  Rows
// flagged NORM_WRITE_OUT are then normed with float32 statistics,
// y = x * rsqrt(mean(x^2) + eps) * gain, and stored in the activation type:
// fragment-packed fp16 / bf16 for the 16-bit MFMA GEMMs (16-byte stores of
// 8-column groups), row-major float32 on the float32 path.  Rows of samples
// that do not run the sub-block are not listed.
#include <type_traits>

#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;

// The segment holding listed row r (segments sorted by prefix): a scan of
// the inline copy with static indices, else a binary search of the table.
__device__ __forceinline__ NormSeg find_seg(const NormArgs& a, int r) {
  if (a.nsegs <= NORM_INLINE_SEGS) {
    NormSeg sg = a.inl[0];
#pragma unroll
    for (int i = 1; i < NORM_INLINE_SEGS; ++i)
      if (i < a.nsegs && a.inl[i].prefix <= r) sg = a.inl[i];
    return sg;
  }
  int lo = 0, hi = a.nsegs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].prefix <= r) lo = mid; else hi = mid - 1;
  }
  return a.segs[lo];
}

// OUT: 0 float32 row-major (float32 gain), 1 bf16 packed, 2 fp16 packed (bf16 gain)
template <int OUT>
__global__ __launch_bounds__(NT) void resid_norm_kernel(NormArgs a) {
  __shared__ float s_part[NT / 64];
  const int r = blockIdx.x;
  const NormSeg sg = find_seg(a, r);
  const size_t row = (size_t)sg.row0 + (r - sg.prefix);
  const size_t prow = (size_t)sg.prow0 + (r - sg.prefix);
  const int D = a.D, tid = threadIdx.x;
  float4* x = reinterpret_cast<float4*>(a.x + row * D);
  const bool add = (sg.flags & NORM_ADD_PARTIALS) != 0;
  float ss = 0.f;
  for (int c = tid; c < D / 4; c += NT) {
    float4 v = x[c];
    if (add) {
      for (int p = 0; p < a.nsplit; ++p) {
        const float4 q = reinterpret_cast<const float4*>(a.partial + p * a.pslice + row * D)[c];
        v.x += q.x; v.y += q.y; v.z += q.z; v.w += q.w;
      }
      x[c] = v;
    }
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  if (!(sg.flags & NORM_WRITE_OUT)) return;   // uniform across the workgroup
  ss = warp_sum(ss);
  if ((tid & 63) == 0) s_part[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) tot += s_part[i];
  const float inv = rsqrtf(tot / (float)D + a.eps);
  if constexpr (OUT != 0) {
    const uint4* gain = reinterpret_cast<const uint4*>(a.gain);
    uint16_t* out = static_cast<uint16_t*>(a.out);
    for (int c = tid; c < D / 8; c += NT) {
      const float4 v0 = x[2 * c], v1 = x[2 * c + 1];
      const uint4 gw = gain[c];
      const float g[8] = {bf16_bits_to_f32(gw.x & 0xffffu), bf16_bits_to_f32(gw.x >> 16),
                          bf16_bits_to_f32(gw.y & 0xffffu), bf16_bits_to_f32(gw.y >> 16),
                          bf16_bits_to_f32(gw.z & 0xffffu), bf16_bits_to_f32(gw.z >> 16),
                          bf16_bits_to_f32(gw.w & 0xffffu), bf16_bits_to_f32(gw.w >> 16)};
      const float y[8] = {v0.x * inv * g[0], v0.y * inv * g[1], v0.z * inv * g[2],
                          v0.w * inv * g[3], v1.x * inv * g[4], v1.y * inv * g[5],
                          v1.z * inv * g[6], v1.w * inv * g[7]};
      const uint4 o = make_uint4(pack_act2<OUT == 2>(y[0], y[1]), pack_act2<OUT == 2>(y[2], y[3]),
                                 pack_act2<OUT == 2>(y[4], y[5]), pack_act2<OUT == 2>(y[6], y[7]));
      const int64_t at = a.rowmajor ? (int64_t)prow * D + 8 * c : packed_index((int64_t)prow, 8 * c, D);
      *reinterpret_cast<uint4*>(out + at) = o;
      if (OUT == 1 && a.out2)
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.out2) + at) =
            make_uint4(bf16_low2(y[0], y[1], o.x), bf16_low2(y[2], y[3], o.y),
                       bf16_low2(y[4], y[5], o.z), bf16_low2(y[6], y[7], o.w));
    }
  } else {
    const float4* gain = reinterpret_cast<const float4*>(a.gain);
    float4* out = reinterpret_cast<float4*>(static_cast<float*>(a.out) + prow * D);
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

// Sets *flag when one of x[0..4 n4) is inf or NaN (x 16-byte aligned);
// every thread that finds one stores the same value.
__global__ void nonfinite_kernel(const float4* x, int64_t n4, uint32_t* flag) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 v = x[i];
    bad = bad || !isfinite(v.x) || !isfinite(v.y) || !isfinite(v.z) || !isfinite(v.w);
  }
  if (bad) *flag = SVL_STATUS_NONFINITE;
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Register-resident variant for D <= 4 * NT * VPT: the row, its pending
// partial slices (four slices per batch of loads) and the gain are loaded
// with every load of a batch in flight at once, the row stays in registers
// for the normed output, and the residual is written back once.  Slices are
// added in slice order, as in the general kernel.
#ifndef SVL_NORM_NT
#define SVL_NORM_NT 1024
#endif
constexpr int NTR = SVL_NORM_NT;   // threads of the one-row-per-workgroup kernel (1024: the
                                   // most loads of the row and its slices in flight at once)

template <int OUT, int VPT>
__global__ __launch_bounds__(NTR) void resid_norm_reg_kernel(NormArgs a) {
  constexpr int NT = NTR;
  __shared__ float s_part[NT / 64];
  const int r = blockIdx.x;
  const NormSeg sg = find_seg(a, r);
  const size_t row = (size_t)sg.row0 + (r - sg.prefix);
  const size_t prow = (size_t)sg.prow0 + (r - sg.prefix);
  const int D4 = a.D >> 2, tid = threadIdx.x;
  float4* x = reinterpret_cast<float4*>(a.x + row * a.D);
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 v[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int c = tid + i * NT;
    v[i] = c < D4 ? x[c] : zero;
  }
  // rows that are normed load the gain with the row (it does not depend on
  // the statistics); add-only launches carry no gain
  const bool write_out = (sg.flags & NORM_WRITE_OUT) != 0;   // uniform across the workgroup
  using GainT = std::conditional_t<OUT != 0, uint2, float4>;
  GainT gv[VPT];
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int c = tid + i * NT;
    gv[i] = write_out && c < D4 ? reinterpret_cast<const GainT*>(a.gain)[c] : GainT{};
  }
  const bool add = (sg.flags & NORM_ADD_PARTIALS) != 0;
  if (add) {
    for (int p0 = 0; p0 < a.nsplit; p0 += 4) {
      float4 q[4][VPT];
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
          const int c = tid + i * NT;
          q[p][i] = (p0 + p < a.nsplit && c < D4)
                        ? reinterpret_cast<const float4*>(a.partial + (p0 + p) * a.pslice + row * a.D)[c]
                        : zero;
        }
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
          v[i].x += q[p][i].x; v[i].y += q[p][i].y; v[i].z += q[p][i].z; v[i].w += q[p][i].w;
        }
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int c = tid + i * NT;
      if (c < D4) x[c] = v[i];
    }
  }
  if (!write_out) return;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < VPT; ++i) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
  ss = warp_sum(ss);
  if ((tid & 63) == 0) s_part[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) tot += s_part[i];
  const float inv = rsqrtf(tot / (float)a.D + a.eps);
#pragma unroll
  for (int i = 0; i < VPT; ++i) {
    const int c = tid + i * NT;
    if (c >= D4) continue;
    if constexpr (OUT != 0) {
      const uint2 gw = gv[i];
      const float g0 = bf16_bits_to_f32(gw.x & 0xffffu), g1 = bf16_bits_to_f32(gw.x >> 16);
      const float g2 = bf16_bits_to_f32(gw.y & 0xffffu), g3 = bf16_bits_to_f32(gw.y >> 16);
      const float y0 = v[i].x * inv * g0, y1 = v[i].y * inv * g1;
      const float y2 = v[i].z * inv * g2, y3 = v[i].w * inv * g3;
      const uint2 o = make_uint2(pack_act2<OUT == 2>(y0, y1), pack_act2<OUT == 2>(y2, y3));
      const int64_t at = a.rowmajor ? (int64_t)prow * a.D + 4 * c
                                    : packed_index((int64_t)prow, 4 * c, a.D);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + at) = o;
      if (OUT == 1 && a.out2)
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out2) + at) =
            make_uint2(bf16_low2(y0, y1, o.x), bf16_low2(y2, y3, o.y));
    } else {
      const float4 g = gv[i];
      reinterpret_cast<float4*>(static_cast<float*>(a.out) + prow * a.D)[c] =
          make_float4(v[i].x * inv * g.x, v[i].y * inv * g.y, v[i].z * inv * g.z, v[i].w * inv * g.w);
    }
  }
}

// Row-group variant for large 16-bit launches: a workgroup takes 8
// consecutive rows of one segment, one wave per row, so the 16-row packed
// layout receives whole 128-byte lines (8 rows x 8 columns) instead of
// 8-byte pieces of one row.  Each wave keeps its row in registers (vpt
// float4 per lane, D = 256 vpt), adds the pending slices in slice order,
// takes the row statistics with a wave reduction, and writes its normed
// values into an LDS staging area whose entry (8-column group kg, row w) sits
// at kg * 144 + w * 16 bytes: the 144-byte stride keeps both the row-wise
// 8-byte writes and the 8-lane line reads on distinct banks.
constexpr int NT8 = 512;
__device__ __forceinline__ NormSeg find_seg8(const NormArgs& a, int g) {
  if (a.nsegs <= NORM_INLINE_SEGS) {
    NormSeg sg = a.inl[0];
#pragma unroll
    for (int i = 1; i < NORM_INLINE_SEGS; ++i)
      if (i < a.nsegs && a.inl[i].gprefix <= g) sg = a.inl[i];
    return sg;
  }
  int lo = 0, hi = a.nsegs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].gprefix <= g) lo = mid; else hi = mid - 1;
  }
  return a.segs[lo];
}

template <int OUT, int VMAX>
__global__ __launch_bounds__(NT8) void resid_norm8_kernel(NormArgs a) {
  static_assert(OUT != 0, "16-bit packed output");
  __shared__ __attribute__((aligned(16))) uint8_t stage[32 * VMAX * 144];
  const int g = blockIdx.x;
  const NormSeg sg = find_seg8(a, g);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int base = (g - sg.gprefix) * 8;          // first local row of the group
  const int local = base + wave;
  const bool valid = local < sg.nrows;            // wave-uniform
  const int vpt = a.D >> 8;
  const size_t row = (size_t)sg.row0 + local;
  float4* x = reinterpret_cast<float4*>(a.x + row * a.D);
  const bool write_out = (sg.flags & NORM_WRITE_OUT) != 0;   // uniform across the workgroup
  float4 v[VMAX];
  uint2 gv[VMAX];
#pragma unroll
  for (int i = 0; i < VMAX; ++i) {
    const int c = lane + 64 * i;
    const bool in = valid && i < vpt;
    v[i] = in ? x[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    gv[i] = in && write_out ? reinterpret_cast<const uint2*>(a.gain)[c] : make_uint2(0u, 0u);
  }
  if (valid && (sg.flags & NORM_ADD_PARTIALS)) {
    for (int p = 0; p < a.nsplit; ++p) {
      const float4* q = reinterpret_cast<const float4*>(a.partial + p * a.pslice + row * a.D);
#pragma unroll
      for (int i = 0; i < VMAX; ++i) {
        if (i >= vpt) continue;
        const float4 t = q[lane + 64 * i];
        v[i].x += t.x; v[i].y += t.y; v[i].z += t.z; v[i].w += t.w;
      }
    }
#pragma unroll
    for (int i = 0; i < VMAX; ++i)
      if (i < vpt) x[lane + 64 * i] = v[i];
  }
  if (!write_out) return;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < VMAX; ++i) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
  ss = warp_sum(ss);
  const float inv = rsqrtf(ss / (float)a.D + a.eps);
  // pass 0: the output; pass 1 (bf16 output with out2): the low parts
  const int npass = (OUT == 1 && a.out2) ? 2 : 1;   // uniform across the workgroup
  for (int pass = 0; pass < npass; ++pass) {
    if (pass) __syncthreads();   // the first pass's pieces are read
    if (valid) {
#pragma unroll
      for (int i = 0; i < VMAX; ++i) {
        if (i >= vpt) continue;
        const int c = lane + 64 * i;                 // columns 4c .. 4c+3
        const uint2 gw = gv[i];
        const float g0 = bf16_bits_to_f32(gw.x & 0xffffu), g1 = bf16_bits_to_f32(gw.x >> 16);
        const float g2 = bf16_bits_to_f32(gw.y & 0xffffu), g3 = bf16_bits_to_f32(gw.y >> 16);
        const float y0 = v[i].x * inv * g0, y1 = v[i].y * inv * g1;
        const float y2 = v[i].z * inv * g2, y3 = v[i].w * inv * g3;
        uint2 o = make_uint2(pack_act2<OUT == 2>(y0, y1), pack_act2<OUT == 2>(y2, y3));
        if (pass) o = make_uint2(bf16_low2(y0, y1, o.x), bf16_low2(y2, y3, o.y));
        *reinterpret_cast<uint2*>(stage + (c >> 1) * 144 + wave * 16 + (c & 1) * 8) = o;
      }
    }
    __syncthreads();
    // piece p: row w = p % 8 of the group, columns 8 (p / 8) .. + 7
    uint16_t* out = static_cast<uint16_t*>(pass ? a.out2 : a.out);
    for (int p = threadIdx.x; p < a.D; p += NT8) {
      const int w = p & 7, kg = p >> 3;
      if (base + w < sg.nrows)
        *reinterpret_cast<uint4*>(out + packed_index((int64_t)sg.prow0 + base + w, 8 * kg, a.D)) =
            *reinterpret_cast<const uint4*>(stage + kg * 144 + w * 16);
    }
  }
}

template <int OUT>
hipError_t launch_norm(const NormArgs& a, hipStream_t st) {
  const int d4 = a.D / 4;
  if constexpr (OUT != 0) {
    if (a.rows8) {
      if (a.D % 256 != 0 || a.D > 8192 || a.ngroups8 <= 0) return hipErrorInvalidValue;
      const int vpt = a.D / 256;
      const unsigned grid = (unsigned)a.ngroups8;
      if (vpt <= 8) resid_norm8_kernel<OUT, 8><<<grid, NT8, 0, st>>>(a);
      else if (vpt <= 16) resid_norm8_kernel<OUT, 16><<<grid, NT8, 0, st>>>(a);
      else resid_norm8_kernel<OUT, 32><<<grid, NT8, 0, st>>>(a);
      return hipGetLastError();
    }
  }
  if (d4 <= NTR) resid_norm_reg_kernel<OUT, 1><<<a.nrows, NTR, 0, st>>>(a);
  else if (d4 <= 2 * NTR) resid_norm_reg_kernel<OUT, 2><<<a.nrows, NTR, 0, st>>>(a);
  else if (d4 <= 4 * NTR) resid_norm_reg_kernel<OUT, 4><<<a.nrows, NTR, 0, st>>>(a);
  else if (d4 <= 8 * NTR) resid_norm_reg_kernel<OUT, 8><<<a.nrows, NTR, 0, st>>>(a);
  else resid_norm_kernel<OUT><<<a.nrows, NT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_resid_norm(const NormArgs& a, int32_t out_kind, hipStream_t st) {
  if (a.nrows <= 0) return hipSuccess;
  if (out_kind == 2) return launch_norm<2>(a, st);
  if (out_kind == 1) return launch_norm<1>(a, st);
  return launch_norm<0>(a, st);
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

hipError_t launch_nonfinite(const float* x, int64_t n, uint32_t* flag, hipStream_t st) {
  const int64_t n4 = n / 4;
  if (n4 <= 0) return hipSuccess;
  const int64_t blocks = (n4 + 255) / 256 < 2048 ? (n4 + 255) / 256 : 2048;
  nonfinite_kernel<<<(unsigned)blocks, 256, 0, st>>>(reinterpret_cast<const float4*>(x), n4, flag);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t value, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  fill_i32_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(p, value, n);
  return hipGetLastError();
}

}  // namespace svl
