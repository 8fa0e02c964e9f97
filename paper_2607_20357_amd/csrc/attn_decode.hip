// KV cache of the decode stage: appending a call's K / V rows, and the
// attention of one new query row per sample over its cached positions.
//
// Cache layout (one layer): [batch][n_kv_heads][2 (K, V)][max_len][d] in the
// activation type; K is stored rotated (the QKV epilogue applies RoPE at each
// row's position).  Only the active K/V heads of samples that run the layer
// are written and read.
//
// Decode attention: one workgroup per (sample, active query head).  The query
// at position p = pos_base attends to positions 0..p: 0..p-1 from the cache,
// p (its own key and value) from the Q/K/V rows of this step, which the
// workgroup of the first active query head of each K/V head also appends to
// the cache for the steps after (no separate append launch in decode).
// Scores are float32 (log2 units, scale folded into q), the softmax is
// max-subtracted, and the probability-weighted values are summed in float32
// per 8-dim group over 16 key partitions, then combined in a fixed order.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;
constexpr int MAX_KEYS = 32768;   // positions one sample's decode attention handles

__device__ __forceinline__ size_t cache_index(const AttnArgs& a, int b, int kvh, int kind,
                                              int pos, int d) {
  return ((((size_t)b * a.n_kv_heads + kvh) * 2 + kind) * (size_t)a.max_len + pos) * d;
}

// grid (max_kv_cnt, ngroups): one workgroup per (sample, active K/V head);
// rows row0 .. row0+S-1 of the Q/K/V buffer go to positions pos_base ..
template <int D>
__global__ __launch_bounds__(NT) void kv_append_kernel(AttnArgs a) {
  const AttnGroup g = a.groups[blockIdx.y];
  const int slot = blockIdx.x;
  if (slot >= g.kv_cnt) return;
  const int kvh = a.kvhead_table[g.kv_off + slot];
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  uint16_t* cache = static_cast<uint16_t*>(a.cache);
  const int kcol = (a.n_heads + kvh) * D, vcol = (a.n_heads + a.n_kv_heads + kvh) * D;
  constexpr int PR = D / 8;   // 16-byte pieces per row
  const int total = g.S * 2 * PR;
  for (int p = threadIdx.x; p < total; p += NT) {
    const int c = p % PR, kind = (p / PR) & 1, i = p / (2 * PR);
    const uint4 v = *reinterpret_cast<const uint4*>(qkv + (size_t)(g.row0 + i) * a.ldq +
                                                    (kind ? vcol : kcol) + 8 * c);
    *reinterpret_cast<uint4*>(cache + cache_index(a, g.sample, kvh, kind, g.pos_base + i, D) +
                              8 * c) = v;
  }
}

template <int NTB>
__device__ __forceinline__ float block_reduce(float v, bool is_max, float* s_red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float u = __shfl_xor(v, o, 64);
    v = is_max ? fmaxf(v, u) : v + u;
  }
  __syncthreads();   // s_red free (an earlier reduction's readers are done)
  if (lane == 0) s_red[w] = v;
  __syncthreads();
  float r = s_red[0];
#pragma unroll
  for (int i = 1; i < NTB / 64; ++i) r = is_max ? fmaxf(r, s_red[i]) : r + s_red[i];
  return r;
}

// 1024 threads: TPK = D / 32 threads per key in the score pass (32 dims each),
// and in the value pass thread t takes dim group t % (D / 8) of the keys
// j = t / (D / 8) (mod NT / (D / 8)); the partitions of a wave are summed with
// shuffles, then the waves' partials in LDS in wave order.
constexpr int NTD = 1024;

template <int D, bool F16>
__global__ __launch_bounds__(NTD) void attn_decode_kernel(AttnArgs a) {
  constexpr int DG = D / 8;           // 8-dim groups of a row
  constexpr int NP = NTD / DG;        // key partitions of the value pass
  constexpr int PW = 64 / DG;         // partitions per wave
  constexpr int TPK = D / 32;         // threads per key in the score pass
  constexpr int KPP = NTD / TPK;      // keys per score pass
  __shared__ float s_p[MAX_KEYS];
  __shared__ float s_q[D];
  __shared__ float s_red[NTD / 64];
  __shared__ float s_o[NTD / 64][D];
  const int t = blockIdx.x;
  if (t >= a.ntiles) return;
  const AttnGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  const int hs = t - g.tile0;
  const int rep = a.n_heads / a.n_kv_heads;
  const int h = a.head_table[g.h_off + hs];
  const int kvh = h / rep;
  const int len = g.pos_base + 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  uint16_t* kcw = static_cast<uint16_t*>(a.cache) + cache_index(a, g.sample, kvh, 0, 0, D);
  uint16_t* vcw = static_cast<uint16_t*>(a.cache) + cache_index(a, g.sample, kvh, 1, 0, D);
  const uint16_t* kc = kcw;
  const uint16_t* vc = vcw;
  const uint16_t* knew = qkv + (size_t)g.row0 * a.ldq + (a.n_heads + kvh) * D;   // position p
  const uint16_t* vnew = qkv + (size_t)g.row0 * a.ldq + (a.n_heads + a.n_kv_heads + kvh) * D;
  // active heads are listed in ascending order, so the heads of one K/V head
  // are adjacent: the first of them appends position p for later steps
  if (hs == 0 || a.head_table[g.h_off + hs - 1] / rep != kvh) {
    if (tid < 2 * (D / 8)) {
      const int c = tid % (D / 8);
      const bool v = tid >= D / 8;
      *reinterpret_cast<uint4*>((v ? vcw : kcw) + (size_t)g.pos_base * D + 8 * c) =
          *reinterpret_cast<const uint4*>((v ? vnew : knew) + 8 * c);
    }
  }
  const float sl2 = a.scale * 1.4426950408889634f;   // scores in log2 units
  // Loads that do not depend on the scores go out first: this thread's key
  // piece of the first score pass and its first NPF value rows, so their
  // latency overlaps the query load, the scores and the softmax.
  const int sub = tid % TPK;
  const int dg = tid % DG, pt = tid / DG;
  constexpr int NPF = 4;
  uint4 kpre[4], vpre[NPF];
  {
    const int j = tid / TPK;
    if (j < len) {
      const uint4* kr = reinterpret_cast<const uint4*>((j == g.pos_base ? knew : kc + (size_t)j * D) + 32 * sub);
#pragma unroll
      for (int c = 0; c < 4; ++c) kpre[c] = kr[c];
    }
#pragma unroll
    for (int i = 0; i < NPF; ++i) {
      const int jv = pt + i * NP;
      vpre[i] = jv < len ? *reinterpret_cast<const uint4*>((jv == g.pos_base ? vnew : vc + (size_t)jv * D) + 8 * dg)
                         : make_uint4(0, 0, 0, 0);
    }
  }
  if (tid < D) s_q[tid] = act_bits_to_f32<F16>(qkv[(size_t)g.row0 * a.ldq + h * D + tid]) * sl2;
  __syncthreads();

  // scores: TPK threads per key, 32 dims each, summed by shuffles
  float mloc = -3.0e38f;
  for (int j0 = 0; j0 < len; j0 += KPP) {
    const int j = j0 + tid / TPK;
    float s = 0.f;
    if (j < len) {
      const uint4* kr = reinterpret_cast<const uint4*>((j == g.pos_base ? knew : kc + (size_t)j * D) + 32 * sub);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint4 v = j0 == 0 ? kpre[c] : kr[c];
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s += act_bits_to_f32<F16>(wv[e] & 0xffffu) * s_q[32 * sub + 8 * c + 2 * e];
          s += act_bits_to_f32<F16>(wv[e] >> 16) * s_q[32 * sub + 8 * c + 2 * e + 1];
        }
      }
    }
#pragma unroll
    for (int o = 1; o < TPK; o <<= 1) s += __shfl_xor(s, o, 64);
    if (j < len) {
      if (sub == 0) s_p[j] = s;
      mloc = fmaxf(mloc, s);
    }
  }
  const float m = block_reduce<NTD>(mloc, true, s_red);
  float lsum = 0.f;
  for (int j = tid; j < len; j += NTD) {
    const float p = exp2f(s_p[j] - m);
    s_p[j] = p;
    lsum += p;
  }
  const float l = block_reduce<NTD>(lsum, false, s_red);   // its barriers also publish s_p

  // values: thread (partition pt, dim group dg) sums keys pt, pt + NP, ...
  // (the first NPF of them from the rows loaded up front)
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < NPF; ++i) {
    const int j = pt + i * NP;
    if (j < len) {
      const float p = s_p[j];
      const uint32_t wv[4] = {vpre[i].x, vpre[i].y, vpre[i].z, vpre[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[2 * e] += p * act_bits_to_f32<F16>(wv[e] & 0xffffu);
        o[2 * e + 1] += p * act_bits_to_f32<F16>(wv[e] >> 16);
      }
    }
  }
#pragma unroll 2
  for (int j = pt + NPF * NP; j < len; j += NP) {
    const uint4 v = *reinterpret_cast<const uint4*>((j == g.pos_base ? vnew : vc + (size_t)j * D) + 8 * dg);
    const float p = s_p[j];
    const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[2 * e] += p * act_bits_to_f32<F16>(wv[e] & 0xffffu);
      o[2 * e + 1] += p * act_bits_to_f32<F16>(wv[e] >> 16);
    }
  }
  // the wave's PW partitions (lanes dg, dg + DG, ...) in a fixed order
#pragma unroll
  for (int e = 0; e < 8; ++e)
#pragma unroll
    for (int sft = DG; sft < 64; sft <<= 1) o[e] += __shfl_xor(o[e], sft, 64);
  if (lane < DG) {
#pragma unroll
    for (int e = 0; e < 8; ++e) s_o[wave][8 * dg + e] = o[e];
  }
  __syncthreads();
  if (tid < DG) {
    const float inv = 1.0f / l;
    float r[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float acc = 0.f;
      for (int q = 0; q < NTD / 64; ++q) acc += s_o[q][8 * tid + e];   // fixed order
      r[e] = acc * inv;
    }
    const uint4 w = make_uint4(pack_act2<F16>(r[0], r[1]), pack_act2<F16>(r[2], r[3]),
                               pack_act2<F16>(r[4], r[5]), pack_act2<F16>(r[6], r[7]));
    // row-major [rows][A d]: the decode step's output projection reads it row by row
    uint16_t* out = static_cast<uint16_t*>(a.out);
    *reinterpret_cast<uint4*>(out + (size_t)g.row0 * a.ldo + h * D + 8 * tid) = w;
  }
  (void)PW;
}

}  // namespace

hipError_t launch_kv_append(const AttnArgs& a, int32_t head_dim, hipStream_t st) {
  if (a.ngroups <= 0 || a.max_kv_cnt <= 0) return hipSuccess;
  const dim3 grid((unsigned)a.max_kv_cnt, (unsigned)a.ngroups);
  if (head_dim == 128) kv_append_kernel<128><<<grid, NT, 0, st>>>(a);
  else if (head_dim == 64) kv_append_kernel<64><<<grid, NT, 0, st>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_decode(const AttnArgs& a, int32_t head_dim, bool f16, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  if (a.max_len > MAX_KEYS) return hipErrorInvalidValue;
  if (head_dim == 128) {
    if (f16) attn_decode_kernel<128, true><<<a.ntiles, NTD, 0, st>>>(a);
    else attn_decode_kernel<128, false><<<a.ntiles, NTD, 0, st>>>(a);
  } else if (head_dim == 64) {
    if (f16) attn_decode_kernel<64, true><<<a.ntiles, NTD, 0, st>>>(a);
    else attn_decode_kernel<64, false><<<a.ntiles, NTD, 0, st>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace svl
