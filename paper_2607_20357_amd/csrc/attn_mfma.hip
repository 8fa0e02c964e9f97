// Causal flash attention over the packed ragged batch, active heads only,
// on 16-bit MFMA (gfx950 v_mfma_f32_16x16x32_{f16,bf16}); Q, K, V, the
// probabilities and the output are fp16 or bf16 (the activation type),
// scores, softmax statistics and accumulators float32.
//
// One workgroup = one (sample, active query head, 64-row query tile); the
// launch lists only active heads, so inactive heads are never read or
// written.  Each of the 4 waves owns 16 query rows.  Scores are formed
// transposed, S^T = K Q^T (kv rows x q columns), so that a lane's
// accumulator entries all belong to one query (q = lane % 16): the softmax
// row statistics stay per lane, and the probabilities already sit in the
// B-operand layout of the next product O^T = V^T P^T.  The k index of that
// product is permuted consistently on both operands (lane group g holds kv
// 4g..4g+3 and 16+4g..16+4g+3 of each 32-row step), which leaves the sum
// unchanged.
//
// Q and K arrive already rotated by RoPE (the QKV projection's epilogue
// rotates them at each row's position inside its sample).  K and V tiles of
// 64 rows go through LDS; V is stored transposed.  The output is written in
// the fragment-packed layout the output projection reads.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BQ = ATTN_BQ, BKV = 64, NT = 256;
constexpr float NEG_BIG = -1.0e30f;

template <int D, bool F16>
__global__ __launch_bounds__(NT) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KS = D + 8;      // K tile row stride (elements)
  constexpr int VS = BKV + 8;    // transposed V tile row stride (elements)
  constexpr int NS = D / 32;     // MFMA k-steps over the head dimension
  constexpr int NB = D / 16;     // 16-wide head-dimension blocks of O^T
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BKV * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VS];

  const int t = blockIdx.x;
  if (t >= a.ntiles) return;
  const AttnGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  const int local = t - g.tile0;
  const int hs = local % g.h_cnt;
  const int qt = g.nqt - 1 - local / g.h_cnt;   // longest query tiles first
  const int h = a.head_table[g.h_off + hs];
  const int kvh = h / (a.n_heads / a.n_kv_heads);
  const int S = g.S, q0 = qt * BQ;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int gq = lane >> 4, lq = lane & 15;
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  const size_t ldq = (size_t)a.ldq;
  const uint16_t* base = qkv + (size_t)g.row0 * ldq;
  const int qcol = h * D, kcol = (a.n_heads + kvh) * D, vcol = (a.n_heads + a.n_kv_heads + kvh) * D;

  // Query fragments: lane holds Q[qi][32 s + 8 gq + j].
  const int qi = q0 + wave * 16 + lq;
  const bool qvalid = qi < S;
  uint4 qf[NS];
  {
    const uint16_t* qp = base + (size_t)(qvalid ? qi : 0) * ldq + qcol;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      uint4 v = *reinterpret_cast<const uint4*>(qp + 32 * s + 8 * gq);
      if (!qvalid) v = make_uint4(0, 0, 0, 0);
      qf[s] = v;
    }
  }

  float m_i = NEG_BIG, l_i = 0.f;
  floatx4 o[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) o[b] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float sl2 = a.scale * 1.4426950408889634f;   // scores in log2 units
  const int kv_end = min(S, q0 + BQ);

  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    // K tile: task = (row, 16-byte chunk).
    for (int task = tid; task < BKV * (D / 8); task += NT) {
      const int row = task / (D / 8), c = task % (D / 8);
      const int kv = kv0 + row;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (kv < S) v = *reinterpret_cast<const uint4*>(base + (size_t)kv * ldq + kcol + 8 * c);
      *reinterpret_cast<uint4*>(&Ks[row * KS + 8 * c]) = v;
    }
    // V tile, transposed: task = (row pair, 8-column chunk).
    for (int task = tid; task < (BKV / 2) * (D / 8); task += NT) {
      const int pr = task / (D / 8), c = task % (D / 8);
      const int kva = kv0 + 2 * pr, kvb = kva + 1;
      uint4 va = make_uint4(0, 0, 0, 0), vb = va;
      if (kva < S) va = *reinterpret_cast<const uint4*>(base + (size_t)kva * ldq + vcol + 8 * c);
      if (kvb < S) vb = *reinterpret_cast<const uint4*>(base + (size_t)kvb * ldq + vcol + 8 * c);
      const uint32_t aw[4] = {va.x, va.y, va.z, va.w}, bw[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = (aw[j] & 0xffffu) | (bw[j] << 16);
        const uint32_t hi = (aw[j] >> 16) | (bw[j] & 0xffff0000u);
        *reinterpret_cast<uint32_t*>(&Vt[(8 * c + 2 * j) * VS + 2 * pr]) = lo;
        *reinterpret_cast<uint32_t*>(&Vt[(8 * c + 2 * j + 1) * VS + 2 * pr]) = hi;
      }
    }
    __syncthreads();

    // S^T = K Q^T for the four 16-row kv blocks.
    floatx4 st[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4 kf = *reinterpret_cast<const uint4*>(&Ks[(16 * i + lq) * KS + 32 * s + 8 * gq]);
        st[i] = mfma16x16x32<F16>(kf, qf[s], st[i]);
      }
    }
    // Causal mask (kv <= q) and online softmax, per query = per lane.
    float mloc = NEG_BIG;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kv = kv0 + 16 * i + 4 * gq + r;
        const float v = (kv <= qi && kv < S) ? st[i][r] * sl2 : NEG_BIG;
        st[i][r] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float m_new = fmaxf(m_i, mloc);
    const float alpha = exp2f(m_i - m_new);
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(st[i][r] - m_new);
        st[i][r] = p;
        lsum += p;
      }
    l_i = l_i * alpha + lsum;
    m_i = m_new;
#pragma unroll
    for (int b = 0; b < NB; ++b) o[b] *= alpha;

    // O^T += V^T P^T, two 32-row kv steps.
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const uint4 pb = make_uint4(pack_act2<F16>(st[2 * t2][0], st[2 * t2][1]),
                                  pack_act2<F16>(st[2 * t2][2], st[2 * t2][3]),
                                  pack_act2<F16>(st[2 * t2 + 1][0], st[2 * t2 + 1][1]),
                                  pack_act2<F16>(st[2 * t2 + 1][2], st[2 * t2 + 1][3]));
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const uint16_t* vr = &Vt[(16 * b + lq) * VS + 32 * t2 + 4 * gq];
        const uint2 v0 = *reinterpret_cast<const uint2*>(vr);
        const uint2 v1 = *reinterpret_cast<const uint2*>(vr + 16);
        o[b] = mfma16x16x32<F16>(make_uint4(v0.x, v0.y, v1.x, v1.y), pb, o[b]);
      }
    }
  }

  l_i += __shfl_xor(l_i, 16, 64);
  l_i += __shfl_xor(l_i, 32, 64);
  if (qvalid) {
    // fragment-packed output for the output projection: the lane's 4
    // consecutive dims 16 b + 4 gq + [0, 4) are contiguous in the layout
    const float inv = 1.0f / l_i;
    uint16_t* out = static_cast<uint16_t*>(a.out);
    const int64_t row = (int64_t)g.row0 + qi;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const uint2 w = make_uint2(pack_act2<F16>(o[b][0] * inv, o[b][1] * inv),
                                 pack_act2<F16>(o[b][2] * inv, o[b][3] * inv));
      *reinterpret_cast<uint2*>(out + packed_index(row, h * D + 16 * b + 4 * gq, a.ldo)) = w;
    }
  }
}

}  // namespace

hipError_t launch_attn_mfma(const AttnArgs& a, int32_t head_dim, bool f16, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  if (head_dim == 128) {
    if (f16) attn_mfma_kernel<128, true><<<a.ntiles, NT, 0, st>>>(a);
    else attn_mfma_kernel<128, false><<<a.ntiles, NT, 0, st>>>(a);
  } else if (head_dim == 64) {
    if (f16) attn_mfma_kernel<64, true><<<a.ntiles, NT, 0, st>>>(a);
    else attn_mfma_kernel<64, false><<<a.ntiles, NT, 0, st>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace svl
