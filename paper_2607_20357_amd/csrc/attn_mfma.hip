// Causal flash attention over the packed ragged batch, active heads only,
// on 16-bit MFMA (gfx950 v_mfma_f32_16x16x32_{f16,bf16}); Q, K, V, the
// probabilities and the output are fp16 or bf16 (the activation type),
// scores, softmax statistics and accumulators float32.
//
// One workgroup = one (sample, active query head, BQ-row query tile); the
// launch lists only active heads, so inactive heads are never read or
// written.  8 waves: with BQ = 64, wave w owns 16 query rows (w % 4) and the
// key tiles of parity w / 4; with BQ = 32 (launches too short to fill the
// chip), wave w owns query rows (w % 2) and the key tiles t with
// t % 4 == w / 2.  Each key partition runs its own online softmax and the
// partitions are combined at the end in partition order, so a query tile's
// key range is walked KP tiles at a time.  Scores are formed
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

constexpr int BKV = 64, NT = 512;
constexpr int GT = 4;   // key tiles loaded together (one LDS buffer each)
constexpr float NEG_BIG = -1.0e30f;

template <int D, bool F16, int BQ>
__global__ __launch_bounds__(NT) void attn_mfma_kernel(AttnArgs a) {
  constexpr int QG = BQ / 16;    // 16-row query groups
  constexpr int KP = 8 / QG;     // key partitions
  static_assert(BQ == 64 || BQ == 32, "query tile of 64 or 32 rows");
  constexpr int KS = D + 8;      // K tile row stride (elements)
  // transposed V tile row stride (elements): 152 bytes.  Measured per launch
  // against strides of 136, 144, 160 and 176 bytes, 152 is fastest (headline
  // 12.6 -> 11.9 us, ragged batch of 8 37.8 -> 33.4 us against 160); every
  // candidate keeps the 8-byte fragment reads and 4-byte stores aligned
  constexpr int VS = BKV + 12;
  constexpr int NS = D / 32;     // MFMA k-steps over the head dimension
  constexpr int NB = D / 16;     // 16-wide head-dimension blocks of O^T
  __shared__ __attribute__((aligned(16))) uint16_t Ks[GT][BKV * KS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[GT][D * VS];

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
  const int qw = wave % QG;      // 16-row query group
  const int part = wave / QG;    // key tiles t with t % KP == part
  const int gq = lane >> 4, lq = lane & 15;
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  const size_t ldq = (size_t)a.ldq;
  const uint16_t* base = qkv + (size_t)g.row0 * ldq;
  const int qcol = h * D, kcol = (a.n_heads + kvh) * D, vcol = (a.n_heads + a.n_kv_heads + kvh) * D;

  // Query fragments: lane holds Q[qi][32 s + 8 gq + j].
  const int qi = q0 + qw * 16 + lq;
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

  // Keys are handled in groups of GT tiles of 64: the group's K and V are
  // loaded into registers all at once (one memory round trip per group;
  // a sequence of up to 256 tokens is a single group), stored into GT LDS
  // buffers, and the next group's loads are issued before the tiles are
  // multiplied.  Buffer loads over the sample's rows (range S rows) read
  // rows past the sample as zero, without branches.
  constexpr int KTASKS = BKV * (D / 8), VTASKS = (BKV / 2) * (D / 8);
  constexpr int KT = (KTASKS + NT - 1) / NT;     // K tile: 16-byte pieces per thread
  constexpr int VT = (VTASKS + NT - 1) / NT;     // V tile: row pairs per thread
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(base), (short)0, (int)((uint32_t)S * (uint32_t)ldq * 2u), 0x00020000);
  uint4 kr[GT][KT], va[GT][VT], vb[GT][VT];
  auto load_group = [&](int g0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < GT; ++j) {
      const int kv0 = g0 + j * BKV;
      if (kv0 >= kv_end) break;   // past the query tile's causal range (uniform)
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const int task = min(tid + i * NT, KTASKS - 1), row = task / (D / 8), c = task % (D / 8);
        kr[j][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
            rs, (uint32_t)((kv0 + row) * ldq + kcol + 8 * c) * 2u, 0, 0));
      }
#pragma unroll
      for (int i = 0; i < VT; ++i) {
        // row pair fastest across lanes: the transposed stores of half a wave
        // are 32 consecutive words
        const int task = min(tid + i * NT, VTASKS - 1), pr = task % (BKV / 2), c = task / (BKV / 2);
        const uint32_t off = (uint32_t)((kv0 + 2 * pr) * ldq + vcol + 8 * c) * 2u;
        va[j][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
        vb[j][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
            rs, off + (uint32_t)ldq * 2u, 0, 0));
      }
    }
  };
  auto store_group = [&](int g0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < GT; ++j) {
      if (g0 + j * BKV >= kv_end) break;   // not loaded, not read
#pragma unroll
      for (int i = 0; i < KT; ++i) {
        const int task = tid + i * NT, row = task / (D / 8), c = task % (D / 8);
        if (KTASKS % NT == 0 || task < KTASKS)
          *reinterpret_cast<uint4*>(&Ks[j][row * KS + 8 * c]) = kr[j][i];
      }
      // V transposed: rows 2pr, 2pr+1 interleaved into 32-bit pairs
#pragma unroll
      for (int i = 0; i < VT; ++i) {
        const int task = tid + i * NT, pr = task % (BKV / 2), c = task / (BKV / 2);
        if (VTASKS % NT != 0 && task >= VTASKS) continue;
        const uint32_t aw[4] = {va[j][i].x, va[j][i].y, va[j][i].z, va[j][i].w};
        const uint32_t bw[4] = {vb[j][i].x, vb[j][i].y, vb[j][i].z, vb[j][i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t lo = (aw[e] & 0xffffu) | (bw[e] << 16);
          const uint32_t hi = (aw[e] >> 16) | (bw[e] & 0xffff0000u);
          *reinterpret_cast<uint32_t*>(&Vt[j][(8 * c + 2 * e) * VS + 2 * pr]) = lo;
          *reinterpret_cast<uint32_t*>(&Vt[j][(8 * c + 2 * e + 1) * VS + 2 * pr]) = hi;
        }
      }
    }
  };
  load_group(0);
  for (int g0 = 0; g0 < kv_end; g0 += GT * BKV) {
    __syncthreads();   // the previous group's readers are done
    store_group(g0);
    __syncthreads();
    if (g0 + GT * BKV < kv_end) load_group(g0 + GT * BKV);
#pragma unroll
    for (int j = 0; j < GT; ++j) {
    const int kv0 = g0 + j * BKV;
    if (kv0 >= kv_end) break;
    if ((kv0 / BKV) % KP != part) continue;   // another partition's tile
    const uint16_t* Kt = Ks[j];
    const uint16_t* Vtt = Vt[j];
    // S^T = K Q^T for the four 16-row kv blocks.
    floatx4 st[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      st[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4 kf = *reinterpret_cast<const uint4*>(&Kt[(16 * i + lq) * KS + 32 * s + 8 * gq]);
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
        // masked keys contribute exactly 0 (a partition may see only masked keys)
        const float p = st[i][r] > 0.5f * NEG_BIG ? exp2f(st[i][r] - m_new) : 0.f;
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
        const uint16_t* vr = &Vtt[(16 * b + lq) * VS + 32 * t2 + 4 * gq];
        const uint2 v0 = *reinterpret_cast<const uint2*>(vr);
        const uint2 v1 = *reinterpret_cast<const uint2*>(vr + 16);
        o[b] = mfma16x16x32<F16>(make_uint4(v0.x, v0.y, v1.x, v1.y), pb, o[b]);
      }
    }
    }
  }

  // Combine the partitions: partitions 1 .. KP-1 hand (m, l, o) to
  // partition 0 through LDS (the K buffers, free after the barrier), which
  // adds them in partition order.
  constexpr int CW = 2 + 4 * NB;   // floats per lane
  static_assert((KP - 1) * QG * 64 * CW * 4 <= (int)sizeof(Ks), "combine buffer");
  float* comb = reinterpret_cast<float*>(&Ks[0][0]);
  __syncthreads();
  if (part > 0) {
    float* c = comb + (((part - 1) * QG + qw) * 64 + lane) * CW;
    c[0] = m_i;
    c[1] = l_i;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) c[2 + 4 * b + r] = o[b][r];
  }
  __syncthreads();
  if (part > 0) return;
  {
    float m = m_i;
#pragma unroll
    for (int p = 1; p < KP; ++p) m = fmaxf(m, comb[((p - 1) * QG + qw) * 64 * CW + lane * CW]);
    const float a0 = exp2f(m_i - m);
    l_i *= a0;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[b][r] *= a0;
#pragma unroll
    for (int p = 1; p < KP; ++p) {
      const float* c = comb + (((p - 1) * QG + qw) * 64 + lane) * CW;
      const float ap = exp2f(c[0] - m);
      l_i += c[1] * ap;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[b][r] += c[2 + 4 * b + r] * ap;
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
  if (a.bq != 64 && a.bq != 32) return hipErrorInvalidValue;
  const bool s32 = a.bq == 32;
  if (head_dim == 128) {
    if (s32) {
      if (f16) attn_mfma_kernel<128, true, 32><<<a.ntiles, NT, 0, st>>>(a);
      else attn_mfma_kernel<128, false, 32><<<a.ntiles, NT, 0, st>>>(a);
    } else {
      if (f16) attn_mfma_kernel<128, true, 64><<<a.ntiles, NT, 0, st>>>(a);
      else attn_mfma_kernel<128, false, 64><<<a.ntiles, NT, 0, st>>>(a);
    }
  } else if (head_dim == 64) {
    if (s32) {
      if (f16) attn_mfma_kernel<64, true, 32><<<a.ntiles, NT, 0, st>>>(a);
      else attn_mfma_kernel<64, false, 32><<<a.ntiles, NT, 0, st>>>(a);
    } else {
      if (f16) attn_mfma_kernel<64, true, 64><<<a.ntiles, NT, 0, st>>>(a);
      else attn_mfma_kernel<64, false, 64><<<a.ntiles, NT, 0, st>>>(a);
    }
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace svl
