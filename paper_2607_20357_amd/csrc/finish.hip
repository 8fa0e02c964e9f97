// Finish of split-K QKV and gate/up launches.
//
// A skinny QKV or gate/up launch may cut K into `nsplit` pieces (so each CU
// streams only part of the activation slice); each piece stores its float32
// accumulators into partial slice p (row stride pld).  These kernels add the
// slices in slice order (a fixed order: results do not depend on scheduling)
// and apply what the fused epilogue applies otherwise:
//   QKV: RoPE of query and key columns at the row's position in its sample,
//     pairs (dim, dim + d/2) of a head; then one rounding to 16 bits into the
//     row-major Q/K/V buffer;
//   SWIGLU: silu(gate) * up of each channel (gate columns, then the up
//     columns at pld / 2), one rounding, stored fragment-packed for the down
//     projection.
// Work items: QKV, 4 rotary pairs of one row (the 8 dims of a 16-column block
// are two items); SWIGLU, 8 channels of one row.  A group's items start at
// MmGroup::fitem0, row-major over (row, block[, half]).
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;

__device__ __forceinline__ float4 add4(float4 a, const float4& b) {
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
  return a;
}

template <bool F16>
__global__ __launch_bounds__(NT) void qkv_finish_kernel(FinishArgs a) {
  const int it = blockIdx.x * NT + threadIdx.x;
  if (it >= a.nitems) return;
  int lo = 0, hi = a.ngroups - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.groups[mid].fitem0 <= it) lo = mid; else hi = mid - 1;
  }
  const MmGroup g = a.groups[lo];
  const int local = it - g.fitem0;
  const int per_row = g.nblocks * 2;
  const int row = local / per_row, rest = local % per_row;
  const int gb = rest >> 1, quad = rest & 1;
  const int d = a.head_dim, half = d >> 1, hb = d >> 4;
  const int dim = (gb % hb) * 8 + quad * 4;            // first rotary index of the item
  const int c1 = g.ocol0 + (gb / hb) * d + dim;        // first-half column; partner c1 + half
  const size_t prow = (size_t)g.orow0 + row;
  float4 x1 = make_float4(0.f, 0.f, 0.f, 0.f), x2 = x1;
  for (int p = 0; p < a.nsplit; ++p) {
    const float* src = a.partial + (size_t)p * a.pslice + prow * a.pld;
    x1 = add4(x1, *reinterpret_cast<const float4*>(src + c1));
    x2 = add4(x2, *reinterpret_cast<const float4*>(src + c1 + half));
  }
  float o1[4] = {x1.x, x1.y, x1.z, x1.w}, o2[4] = {x2.x, x2.y, x2.z, x2.w};
  if (g.rope) {
    const float2* cs = a.rope + (size_t)(g.pos_base + row) * half + dim;   // position of the row
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float2 c = cs[i];
      const float u = o1[i], v = o2[i];
      o1[i] = u * c.x - v * c.y;
      o2[i] = v * c.x + u * c.y;
    }
  }
  uint16_t* out = static_cast<uint16_t*>(a.out) + prow * a.ldo;
  *reinterpret_cast<uint2*>(out + c1) = make_uint2(pack_act2<F16>(o1[0], o1[1]), pack_act2<F16>(o1[2], o1[3]));
  *reinterpret_cast<uint2*>(out + c1 + half) =
      make_uint2(pack_act2<F16>(o2[0], o2[1]), pack_act2<F16>(o2[2], o2[3]));
}

template <bool F16>
__global__ __launch_bounds__(NT) void swiglu_finish_kernel(FinishArgs a) {
  const int it = blockIdx.x * NT + threadIdx.x;
  if (it >= a.nitems) return;
  int lo = 0, hi = a.ngroups - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.groups[mid].fitem0 <= it) lo = mid; else hi = mid - 1;
  }
  const MmGroup g = a.groups[lo];
  const int local = it - g.fitem0;
  const int row = local / g.nblocks, gb = local % g.nblocks;
  const int ch = g.ocol0 + gb * 8;
  const size_t prow = (size_t)g.orow0 + row;
  const int up_off = a.pld >> 1;
  float4 g0 = make_float4(0.f, 0.f, 0.f, 0.f), g1 = g0, u0 = g0, u1 = g0;
  for (int p = 0; p < a.nsplit; ++p) {
    const float* src = a.partial + (size_t)p * a.pslice + prow * a.pld + ch;
    g0 = add4(g0, *reinterpret_cast<const float4*>(src));
    g1 = add4(g1, *reinterpret_cast<const float4*>(src + 4));
    u0 = add4(u0, *reinterpret_cast<const float4*>(src + up_off));
    u1 = add4(u1, *reinterpret_cast<const float4*>(src + up_off + 4));
  }
  const float gt[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float up[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
  float h[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) h[i] = gt[i] / (1.0f + __expf(-gt[i])) * up[i];
  const uint4 o = make_uint4(pack_act2<F16>(h[0], h[1]), pack_act2<F16>(h[2], h[3]),
                             pack_act2<F16>(h[4], h[5]), pack_act2<F16>(h[6], h[7]));
  *reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.out) + packed_index((int64_t)prow, ch, a.ldo)) = o;
}

}  // namespace

hipError_t launch_finish(const FinishArgs& a, int32_t epi, bool f16, hipStream_t st) {
  if (a.nitems <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((a.nitems + NT - 1) / NT);
  if (epi == EPI_QKV) {
    if (f16) qkv_finish_kernel<true><<<grid, NT, 0, st>>>(a);
    else qkv_finish_kernel<false><<<grid, NT, 0, st>>>(a);
  } else if (epi == EPI_SWIGLU) {
    if (f16) swiglu_finish_kernel<true><<<grid, NT, 0, st>>>(a);
    else swiglu_finish_kernel<false><<<grid, NT, 0, st>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace svl
