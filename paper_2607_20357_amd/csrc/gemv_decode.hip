// Row-vector products of the decode step.
//
// In a decode step every GEMM group holds one row: the new token of one
// sample.  Such a launch is a list of 16-column weight blocks (the same
// blocks the MFMA tiles are cut into: QKV blocks pair 8 dims of a head with
// their rotary partners, gate/up blocks pair 8 gate channels with the same 8
// up channels), and its time is the time to stream the blocks' weight rows.
// Four workgroups per block, 4 waves each: a wave computes one column of the
// block, the dot product of one weight row with the sample's activation row
// over the group's K chunks; a workgroup holds two columns and their pair
// partners.  Activation rows are row-major in decode (the norm,
// the decode attention and this kernel's SwiGLU output write them so): a
// row of the fragment-packed layout would be spread over eight cache lines
// per 64 columns.  Lane l takes 8 consecutive columns of chunk
// 8 s + l / 8 in step s; four steps are loaded before they are used, so a
// wave keeps 4 KiB of its weight row in flight.  The lane sums are reduced
// in a fixed order and a workgroup's 4 results meet in LDS for the paired
// epilogues: RoPE on query / key columns, silu(gate) * up, or the residual
// add of the output and down projections (one writer per element).
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int GV_WAVES = 4, GV_NT = GV_WAVES * 64, GV_U = 4;

// Workgroup x takes quarter q = x % 4 of block x / 4: columns 2q, 2q + 1 and
// their partners 2q + 8, 2q + 9 (wave w: column (w & 1) + 2q + 8 (w >> 1)).
constexpr int GV_MAX_CHUNKS = 1024;   // K chunks of a group (K <= 65536)

template <int EPI, bool F16>
__global__ __launch_bounds__(GV_NT) void gemv_kernel(MmArgs a) {
  __shared__ float s_v[GV_WAVES];
  __shared__ int32_t s_k0[GV_MAX_CHUNKS];   // a chunk-list group's offsets (no dependent loads)
  const int blk = blockIdx.x >> 2, quarter = blockIdx.x & 3;
  int lo = 0, hi = a.ngroups - 1;   // the group whose first block (pad0) is the largest <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.groups[mid].pad0 <= blk) lo = mid; else hi = mid - 1;
  }
  const MmGroup g = a.groups[lo];
  const int gb = blk - g.pad0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ci = (wave & 1) + 2 * quarter + ((wave >> 1) ? 8 : 0);
  const int d = a.head_dim, hb = d >> 4, half = d >> 1;
  int m, row;
  if constexpr (EPI == EPI_QKV) {
    m = g.wsel;
    row = g.wrow0 + (gb / hb) * d + (gb % hb) * 8 + (ci & 7) + ((ci >> 3) ? half : 0);
  } else if constexpr (EPI == EPI_SWIGLU) {
    m = ci >> 3;   // gate rows, then up rows
    row = g.wrow0 + gb * 8 + (ci & 7);
  } else {
    m = 0;
    row = g.wrow0 + gb * 16 + ci;
  }
  const uint16_t* wr =
      static_cast<const uint16_t*>(m == 0 ? a.W[0] : (m == 1 ? a.W[1] : a.W[2])) + (size_t)row * a.ldw;
  const uint16_t* xr = static_cast<const uint16_t*>(a.A) + (size_t)g.arow0 * a.lda;
  const int nc = g.kc_cnt, cl = lane >> 3, off = (lane & 7) * 8;
  const bool dense = g.kdense >= 0;   // uniform across the workgroup
  if (!dense) {
    // chunk-list groups (output / down projections under head or FFN gates)
    // cover whole 64-column chunks: runs of heads (d in {64, 128}) and FFN
    // slices (a multiple of 64)
    for (int c = threadIdx.x; c < nc; c += GV_NT) s_k0[c] = a.chunks[g.kc_off + c].k0;
    __syncthreads();
  }
  float acc = 0.f;
  for (int s0 = 0; s0 < nc; s0 += 8 * GV_U) {
    uint4 wv[GV_U], xv[GV_U];
#pragma unroll
    for (int u = 0; u < GV_U; ++u) {
      const int c = s0 + 8 * u + cl;
      if (c < nc) {
        const int k = (dense ? g.kdense + MFMA_BK * c : s_k0[c]) + off;
        wv[u] = *reinterpret_cast<const uint4*>(wr + k);
        xv[u] = *reinterpret_cast<const uint4*>(xr + k);
      } else {
        wv[u] = make_uint4(0, 0, 0, 0);
        xv[u] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < GV_U; ++u) {
      const uint32_t w4[4] = {wv[u].x, wv[u].y, wv[u].z, wv[u].w};
      const uint32_t x4[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc += bf16_bits_to_f32(w4[e] & 0xffffu) * act_bits_to_f32<F16>(x4[e] & 0xffffu);
        acc += bf16_bits_to_f32(w4[e] >> 16) * act_bits_to_f32<F16>(x4[e] >> 16);
      }
    }
  }
  acc = warp_sum(acc);
  if (lane == 0) s_v[wave] = acc;
  __syncthreads();
  if (lane != 0) return;
  float v = s_v[wave];
  if constexpr (EPI == EPI_QKV) {
    const int dim = (gb % hb) * 8 + (ci & 7);
    const int col = g.ocol0 + (gb / hb) * d + dim + ((ci >> 3) ? half : 0);
    if (g.rope) {
      // (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin); columns ci < 8 hold x1
      const float pv = s_v[wave ^ 2];
      const float2 cs = a.rope[(size_t)g.pos_base * half + dim];
      v = v * cs.x + ((ci < 8) ? -pv : pv) * cs.y;
    }
    static_cast<uint16_t*>(a.out)[(size_t)g.orow0 * a.ldo + col] = f32_to_act_bits<F16>(v);
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (ci < 8) {
      const float up = s_v[wave + 2];
      const float h = v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)) * up;
      static_cast<uint16_t*>(a.out)[(size_t)g.orow0 * a.ldo + g.ocol0 + gb * 8 + ci] =
          f32_to_act_bits<F16>(h);
    }
  } else {
    float* o = static_cast<float*>(a.out) + (size_t)g.orow0 * a.ldo + g.ocol0 + gb * 16 + ci;
    *o += v;
  }
}

template <bool F16>
hipError_t launch(const MmArgs& a, int32_t epi, hipStream_t st) {
  const unsigned grid = (unsigned)a.nblocks * 4;
  switch (epi) {
    case EPI_QKV: gemv_kernel<EPI_QKV, F16><<<grid, GV_NT, 0, st>>>(a); break;
    case EPI_SWIGLU: gemv_kernel<EPI_SWIGLU, F16><<<grid, GV_NT, 0, st>>>(a); break;
    case EPI_RESID: gemv_kernel<EPI_RESID, F16><<<grid, GV_NT, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemv(const MmArgs& a, int32_t epi, bool f16, hipStream_t st) {
  if (a.nblocks <= 0 || a.ngroups <= 0) return hipSuccess;
  if (a.lda / MFMA_BK > GV_MAX_CHUNKS) return hipErrorInvalidValue;
  return f16 ? launch<true>(a, epi, st) : launch<false>(a, epi, st);
}

}  // namespace svl
