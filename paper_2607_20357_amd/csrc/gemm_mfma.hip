// Masked grouped GEMM on 16-bit MFMA (gfx950 v_mfma_f32_16x16x32_{f16,bf16}).
//
//   C[rows, cols] = sum over the tile's K chunks of A[rows, k] * W[cols, k]
//
// A is an activation matrix in the fragment-packed layout (plan_types.h:
// 16-row x 64-column blocks of 2 KB, fp16 or bf16); W a bf16 weight matrix
// in [out][in] layout.  With fp16 activations each weight tile is widened
// bf16 -> fp16 on its way into LDS (exact inside fp16's range), so both
// operands of the fp16 MFMA carry 11-bit significands; with bf16 activations
// the weights go through unchanged.  Accumulation is float32.
//
// The launch is a table of tiles built on the host.  A group is one sample
// and one active column range (QKV: a run of active heads of one of Q, K, V;
// gate/up: a run of active FFN slices; output / down projections: all
// columns, with K restricted to the active heads' / slices' columns), so
// weight rows and columns of inactive heads and FFN slices are never read.
// In a batch, a QKV or gate/up group covers a run of consecutive samples
// that all use its heads or slices (their padded rows are contiguous; the
// padding rows between them compute values nobody reads), and its RoPE
// positions come from a per-row table.
// A tile is up to 256 rows of a group times nblk <= NB 16-column blocks
// times a range of K chunks; the planner balances the block counts so a
// launch has about one tile per CU (every tile streams the whole activation
// slice it multiplies, so a launch with fewer, wider tiles reads less).
//
// Workgroup: 512 threads = 8 waves, wave w owning tile rows 32w .. 32w+31
// (two 16-row MFMA blocks) and all blocks of the tile; or, for launches
// with more tiles than CUs (the output / down projections), 256 threads =
// 4 waves of four 16-row blocks each, two workgroups per CU.  K advances in
// chunks of 64.  Per chunk:
//   * each wave loads its own A fragments straight from the packed layout
//     into registers (two 1 KB contiguous loads per 16-row block);
//   * the tile's weight rows are loaded cooperatively (16 bytes per thread
//     and row segment) and staged through LDS, where all waves read them.
// The weights are staged KS = 4 chunks at a time (one barrier per stage,
// so the waves drift freely inside a stage), double-buffered in LDS with one
// or two further stages in flight in registers; A runs 4 (8 waves) or 2
// (4 waves) chunks ahead.
// Loads are buffer loads whose range ends at the last valid row, so rows
// past the tile read as zero.
//
// Epilogues:
//   QKV (paired): RoPE at the row's position inside its sample is applied to
//     the float32 accumulators of query and key groups (partner value from
//     lane ^ 8), then the 16-bit result is stored row-major;
//   SWIGLU (paired): silu(gate) * up, stored fragment-packed for the down
//     projection;
//   RESID (plain): added into the float32 residual;
//   PARTIAL (plain): split-K piece stored into its float32 partial slice; the
//     next residual-finish kernel adds the slices in slice order.
#include <type_traits>
#include <utility>

#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BM = MFMA_BM;
#ifndef SVL_GEMM_KS
#define SVL_GEMM_KS 4
#endif
constexpr int KS = SVL_GEMM_KS;                // K chunks per weight stage (one barrier each)
constexpr int LDS_STRIDE = KS * MFMA_BK;       // 16-bit elements per LDS row (512 B, 32 units)
constexpr int MAX_CHUNKS = 1024;               // K chunks per tile (K <= 65536)
#ifndef SVL_GEMM_NSA
#define SVL_GEMM_NSA KS
#endif
constexpr int NSA8 = SVL_GEMM_NSA;             // A chunks in flight, 8-wave tiles

// Raw buffer resource over [p, p + bytes): loads past the end return zero.
// The inputs are wave-uniform; readfirstlane keeps the descriptor in scalar
// registers even where the compiler cannot prove it (a descriptor it takes
// for divergent costs a loop over lanes at every load).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint64_t ua = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(a >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(ua), (short)0,
                                           __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000);
}

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// LDS row swizzle.  gfx950's LDS serves a 16-byte-per-lane access half a
// wave at a time, 512 bytes over 128 four-byte banks, so the 32 lanes must
// hit 32 distinct 16-byte units modulo 32.  A weight row of a stage is 32
// units (4 chunks x 8); unit v of tile row r is stored at v ^ swz(r).  The
// fragment reads (16 rows x lane groups 0, 1 or 2, 3) and the stores (one
// row's 32 units per half wave) are then conflict-free.
__device__ __forceinline__ int swz(int r) { return (r & 1) | (((r >> 1) & 7) << 2); }

// Weights are streamed once: non-temporal loads.
__device__ __forceinline__ uint4 load16w(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 2));
}

template <bool F16>
__device__ __forceinline__ uint4 weight_to_act(const uint4& v) {
  if constexpr (F16) {
    return make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z),
                      bf16x2_to_f16x2(v.w));
  } else {
    return v;
  }
}

template <int P>
using Phase = std::integral_constant<int, P>;

// NWAVE waves per workgroup, each RB 16-row blocks of the tile: 8 x 2 (two
// waves per SIMD), or 4 x 4 (one wave per SIMD; each LDS operand feeds twice
// the MFMAs, the accumulators sit in the AGPRs, and two workgroups share a
// CU: the output / down projections of launches with more tiles than CUs).
// HILO (bf16 products of QKV / gate-up): every A fragment comes with its low
// bf16 part from A2, multiplied right after it against the same weight
// fragment, so the activations enter the products with about 16 significant
// bits.
template <int EPI, int NB, bool F16, int NWAVE, bool HILO = false>
__global__ __launch_bounds__(NWAVE * 64) void gemm_mfma_kernel(MmArgs a) {
  constexpr int NT = NWAVE * 64;
  constexpr int RB = BM / (16 * NWAVE);         // 16-row blocks per wave
  static_assert(RB * 16 * NWAVE == BM, "waves cover the tile's rows");
  constexpr int BN = NB * 16;                   // weight rows per tile
  // gate/up: weight loads of the next stage issued before the stage barrier
  // (measured 2.8 us faster per headline launch; the other epilogues' shapes
  // measured slightly slower with it)
  constexpr bool EARLY_W = EPI == EPI_SWIGLU;
#ifdef SVL_GEMM_NWS
  constexpr int NWS = SVL_GEMM_NWS;
#else
  constexpr int NWS = NB <= (NWAVE == 8 ? 6 : 3) ? 2 : 1;   // weight register stages
#endif
  static_assert(!HILO || (!F16 && NWAVE == 8), "low parts: bf16 products, 8-wave tiles");
  // A chunks in flight (register slot = chunk % NSA); with the low terms the
  // tiles of up to 4 blocks keep four within the registers (211-256 VGPRs,
  // 5.60 -> 5.30-5.52 ms per bf16 headline step), wider ones two
  constexpr int NSA = HILO ? (NB <= 4 ? 4 : 2) : (NWAVE == 8 ? NSA8 : 2);
  constexpr int AU = HILO ? 4 : 2;              // A fragments per row block and chunk
  static_assert(KS % NSA == 0, "a stage holds whole rounds of A slots");
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2 * BN * LDS_STRIDE];
  __shared__ int32_t s_k0[MAX_CHUNKS];          // the tile's chunk offsets (no vmcnt waits)

  const int t = xcd_tile_index();
  if (t >= a.ntiles) return;
  const MmTile tl = a.tiles[t];
  const int mcnt = tl.mcnt;
  const int nblk = tl.nblk;
  const int nk = tl.kcn;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tl.kdense >= 0) {
    for (int c = tid; c < nk; c += NT) s_k0[c] = tl.kdense + MFMA_BK * c;
  } else {
    for (int c = tid; c < nk; c += NT) s_k0[c] = a.chunks[tl.chunk0 + c].k0;
  }

  const int d = a.head_dim, hb = d >> 4;        // QKV: blocks per head

  // A: packed blocks of this tile's rows; wave w reads 16-row blocks RB w .. RB w + RB-1.
  const uint32_t kblocks = (uint32_t)(a.lda / 64);
  const uint32_t blk_bytes = kblocks * 2048u;   // one 16-row block over all of K
  const int rb0 = (tl.arow) / 16;
  const __amdgpu_buffer_rsrc_t rsA =
      make_rsrc(static_cast<const uint16_t*>(a.A) + (size_t)rb0 * kblocks * 1024,
                (uint32_t)((mcnt + 15) / 16) * blk_bytes);
  const __amdgpu_buffer_rsrc_t rsA2 =
      make_rsrc(static_cast<const uint16_t*>(HILO ? a.A2 : a.A) + (size_t)rb0 * kblocks * 1024,
                HILO ? (uint32_t)((mcnt + 15) / 16) * blk_bytes : 0u);
  uint32_t voA[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) voA[i] = (uint32_t)(RB * wave + i) * blk_bytes + lane * 16u;
  bool rowblk[RB];   // this wave's 16-row blocks hold rows of the tile (wave-uniform)
#pragma unroll
  for (int i = 0; i < RB; ++i) rowblk[i] = 16 * (RB * wave + i) < mcnt;

  // Weights, one stage = KS chunks: piece p = tid + NT*s (s < WLD) is unit
  // p % 32 (chunk u / 8 of the stage, 16-byte segment u % 8) of tile row
  // p / 32 (block j = row/16, column i = row%16 of the block).  Half a wave
  // loads 512 bytes of one weight row; a wave's two rows share one column
  // half of a block (i < 8 or i >= 8), so the matrix choice is wave-uniform.
  static_assert(KS == 4 || KS == 8, "stage rows are 512 or 1024 bytes");
  constexpr int RU = KS * 8;                    // 16-byte units per stage row
  constexpr int WLD = BN * RU / NT;             // BN * RU pieces / NT threads
  static_assert(BN * RU % NT == 0, "whole weight pieces per thread");
  __amdgpu_buffer_rsrc_t rsB[WLD];
  uint32_t voB[WLD];
  const int wu = tid & (RU - 1), wqc = wu >> 3;   // this thread's unit and chunk of the stage
#pragma unroll
  for (int s = 0; s < WLD; ++s) {
    const int tr = (tid + NT * s) / RU;
    const int j = tr >> 4, i = tr & 15;
    const int gb = tl.b0 + j;
    int m = 0, row = 0;
    if constexpr (EPI == EPI_QKV) {
      m = tl.wsel;
      row = tl.wrow0 + (gb / hb) * d + (gb % hb) * 8 + (i & 7) + ((i >> 3) ? (d >> 1) : 0);
    } else if constexpr (EPI == EPI_SWIGLU) {
      m = __builtin_amdgcn_readfirstlane((i >> 3) & 1);   // gate rows, then up rows
      row = tl.wrow0 + gb * 8 + (i & 7);
    } else {
      m = 0;
      row = tl.wrow0 + gb * 16 + i;
    }
    const void* base = m == 0 ? a.W[0] : (m == 1 ? a.W[1] : a.W[2]);
    const int rows = m == 0 ? a.w_rows[0] : (m == 1 ? a.w_rows[1] : a.w_rows[2]);
    rsB[s] = make_rsrc(base, (uint32_t)rows * (uint32_t)a.ldw * 2u);
    // pieces past the tile's blocks read out of range (zero, no traffic); the
    // chunk offset added later (< 2^17) keeps 2^31 out of range without
    // wrapping (a weight matrix spans less than 2^31 bytes)
    voB[s] = j < nblk ? (uint32_t)row * a.ldw * 2u + (wu & 7) * 16u : 0x80000000u;
  }
  __syncthreads();   // s_k0 ready

  const int last = nk - 1;
  uint4 sa[NSA][RB][AU], sw[NWS][WLD];
  // A loads and MFMAs of the wave's NRB row blocks that hold rows of the
  // tile (the pipeline is instantiated per NRB, so a wave past the tile's
  // rows issues no loads for them and the waits stay exact).  NRB < 0: all RB
  // blocks are loaded (out-of-range rows read zero) and the MFMAs branch on
  // rowblk, which keeps the widest tiles within the registers.
  auto loadA = [&](auto nrb, int c, uint4 (&ra)[RB][AU]) __attribute__((always_inline)) {
    constexpr int NRB = decltype(nrb)::value < 0 ? RB : decltype(nrb)::value;
    const uint32_t soA = (uint32_t)__builtin_amdgcn_readfirstlane(s_k0[c]) * 32u;
#pragma unroll
    for (int i = 0; i < NRB; ++i) {
      ra[i][0] = load16(rsA, voA[i], soA);
      ra[i][1] = load16(rsA, voA[i] + 1024u, soA);
      if constexpr (HILO) {
        ra[i][2] = load16(rsA2, voA[i], soA);
        ra[i][3] = load16(rsA2, voA[i] + 1024u, soA);
      }
    }
  };
  // weight stage S: chunks S*KS .. S*KS + KS-1 (past the last: the last again);
  // the chunk offset varies across the half wave, so it goes in the lane offset
  auto loadW = [&](int S, uint4 (&rb)[WLD]) __attribute__((always_inline)) {
    const uint32_t ko = (uint32_t)s_k0[min(S * KS + wqc, last)] * 2u;
#pragma unroll
    for (int s = 0; s < WLD; ++s) rb[s] = load16w(rsB[s], voB[s] + ko, 0);
  };
  auto wstore = [&](int buf, const uint4 (&rb)[WLD]) __attribute__((always_inline)) {
    uint16_t* B = Bs + buf * (BN * LDS_STRIDE);
#pragma unroll
    for (int s = 0; s < WLD; ++s) {
      const int tr = (tid + NT * s) / RU;
      *reinterpret_cast<uint4*>(&B[tr * LDS_STRIDE + (wu ^ swz(tr)) * 8]) =
          weight_to_act<F16>(rb[s]);
    }
  };

  floatx4 acc[RB][NB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Inside a chunk, lane group q = lane / 16 holds k 16q + [0, 8) in the
  // first MFMA k-step and 16q + [8, 16) in the second, for both operands.
  // fragment unit of lane group g in chunk q, k-step ks: q*8 + 2g + ks; the
  // swizzle of rows j*16 + lane%16 depends on lane%16 only
  const int fl = (2 * (lane >> 4)) ^ swz(lane & 15);
  const uint16_t* Bl = Bs + (lane & 15) * LDS_STRIDE;
  auto compute = [&](auto nrb, int buf, int q, const uint4 (&ra)[RB][AU]) __attribute__((always_inline)) {
    constexpr bool DYN = decltype(nrb)::value < 0;
    constexpr int NRB = DYN ? RB : decltype(nrb)::value;
    const uint16_t* B = Bl + buf * (BN * LDS_STRIDE);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 bfr[NB];
      const int u = ((q * 8 + ks) ^ fl) * 8;
      // Blocks past the tile's nblk hold zero weights (their loads read out
      // of range), so they are multiplied unconditionally: straight-line code
      // lets the compiler overlap the LDS reads with the MFMAs.
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bfr[j] = *reinterpret_cast<const uint4*>(&B[j * 16 * LDS_STRIDE + u]);
#pragma unroll
      for (int i = 0; i < NRB; ++i)
        if (!DYN || rowblk[i])
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            acc[i][j] = mfma16x16x32<F16>(ra[i][ks], bfr[j], acc[i][j]);
            if constexpr (HILO) acc[i][j] = mfma16x16x32<F16>(ra[i][2 + ks], bfr[j], acc[i][j]);
          }
    }
  };

  // Pipeline.  Weight stage S (KS chunks) is multiplied from LDS buffer S % 2
  // while stages S+1 .. S+NWS are in flight in registers; chunk c's A
  // fragments sit in register slot c % NSA, loaded NSA chunks ahead.  After
  // stage S: stage S+1 goes from registers into the other LDS buffer, one
  // barrier, and the register stage is refilled with stage S+1+NWS.  Waves
  // synchronise once per KS chunks.
  auto pipeline = [&](auto nrb) __attribute__((always_inline)) {
    const int nst = (nk + KS - 1) / KS;
    // first weight stage and first A chunk ahead of the rest, so the first
    // MFMAs wait for those alone
    loadW(0, sw[0]);
    loadA(nrb, 0, sa[0]);
#pragma unroll
    for (int s = 1; s < NWS; ++s) loadW(s, sw[s]);
    [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
      ((Q > 0 ? loadA(nrb, min(Q, last), sa[Q]) : void()), ...);
    }(std::make_integer_sequence<int, NSA>{});
    wstore(0, sw[0]);
    loadW(NWS, sw[0]);
    __syncthreads();
    // FULL: the stage has KS chunks and a successor (no checks, so the
    // compiler's waits count exactly the loads issued since).
    auto stage = [&](int S, auto ph, auto full) __attribute__((always_inline)) {
      constexpr int P = decltype(ph)::value;   // S % NWS
      constexpr bool FULL = decltype(full)::value;
      [&]<int... Q>(std::integer_sequence<int, Q...>) __attribute__((always_inline)) {
        ((FULL || S * KS + Q < nk
              ? (compute(nrb, S & 1, Q, sa[Q % NSA]),
                 loadA(nrb, min(S * KS + Q + NSA, last), sa[Q % NSA]))
              : void()),
         ...);
      }(std::make_integer_sequence<int, KS>{});
      if (FULL || S + 1 < nst) {
        wstore((S + 1) & 1, sw[(P + 1) % NWS]);
        if constexpr (EARLY_W) {
          // refill the register stage before the barrier: a wave's next
          // weight loads do not wait for the slowest wave
          loadW(S + 1 + NWS, sw[(P + 1) % NWS]);
          __syncthreads();
        } else {
          __syncthreads();
          loadW(S + 1 + NWS, sw[(P + 1) % NWS]);
        }
      }
    };
    const int nmain = min(nk / KS, nst - 1);   // full stages with a successor
    int S = 0;
    for (; S + NWS <= nmain; S += NWS)
      [&]<int... P>(std::integer_sequence<int, P...>) __attribute__((always_inline)) {
        (stage(S + P, Phase<P>{}, std::true_type{}), ...);
      }(std::make_integer_sequence<int, NWS>{});
    // at most NWS + 1 stages remain
    [&]<int... P>(std::integer_sequence<int, P...>) __attribute__((always_inline)) {
      ((S + P < nst ? stage(S + P, Phase<P % NWS>{}, std::false_type{}) : void()), ...);
    }(std::make_integer_sequence<int, NWS + 1>{});
  };
  // every instantiation runs the same barrier sequence
  if (nk > 0) {
    if constexpr (NB >= 8 || NWAVE != 8) {
      pipeline(std::integral_constant<int, -1>{});
    } else {
      if (rowblk[1]) pipeline(std::integral_constant<int, 2>{});
      else if (rowblk[0]) pipeline(std::integral_constant<int, 1>{});
      else pipeline(std::integral_constant<int, 0>{});
    }
  }

  // Epilogue.  acc[i][j][r] is C[16 RB wave + 16 i + 4 (lane/16) + r][16 j + lane%16]
  // of the tile; tile row m is row m0 + m of the group.
  const int rbase = wave * 16 * RB + (lane >> 4) * 4;
  const int ci = lane & 15;           // column inside the block
  if constexpr (EPI == EPI_QKV || EPI == EPI_SWIGLU) {
    if (a.split > 1) {
      // split-K piece: raw float32 accumulators at the output column (QKV) or
      // at the gate / up column (SWIGLU); the finish kernel does the rest
      float* out = a.partial + (size_t)tl.slice * a.pslice;
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rbase + 16 * i + r;
          float* orow = out + (size_t)(tl.orow + min(row, mcnt - 1)) * a.pld;
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const int gb = tl.b0 + j;
            int col;
            if constexpr (EPI == EPI_QKV)
              col = tl.ocol0 + (gb / hb) * d + (gb % hb) * 8 + (ci & 7) + ((ci >> 3) ? (d >> 1) : 0);
            else
              col = ((ci >> 3) ? (a.pld >> 1) : 0) + tl.ocol0 + gb * 8 + (ci & 7);
            if (j < nblk && row < mcnt) orow[col] = acc[i][j][r];
          }
        }
      return;
    }
  }
  if constexpr (EPI == EPI_QKV || EPI == EPI_SWIGLU) {
    // 16-bit outputs go through a per-wave staging tile in the (now idle)
    // weight buffers, 32 rows x RW values: QKV, both halves of every block
    // (16 NB columns); SWIGLU, the 8 NB channels.  Each lane then stores
    // whole 16-byte pieces (8 consecutive columns of one row), instead of
    // one 2-byte value per row and block.
    // (SWIGLU rows are padded to an odd number of 16-byte pieces, so the
    // row-strided piece reads below hit distinct banks)
    constexpr int RW = EPI == EPI_QKV ? NB * 16 : (NB | 1) * 8;
    static_assert(NWAVE * 16 * RB * RW <= 2 * BN * LDS_STRIDE, "staging tiles fit the weight buffers");
    uint16_t* E = Bs + wave * (16 * RB * RW);
    const int lr0 = (lane >> 4) * 4;    // wave-local row of acc[i][j][0] is lr0 + 16 i
    uint16_t* out = static_cast<uint16_t*>(a.out);
    if constexpr (EPI == EPI_QKV) {
      const int half = d >> 1;
      // all table loads before the barrier and the stores
      float2 cs[RB][4][NB];
      if (tl.rope) {
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int rr = min(rbase + 16 * i + r, mcnt - 1);
            const int pos = tl.pos0 >= 0 ? tl.pos0 + rr : a.rowpos[tl.arow + rr];
#pragma unroll
            for (int j = 0; j < NB; ++j) {
              const int gb = tl.b0 + min(j, nblk - 1);
              const int dim = (gb % hb) * 8 + (ci & 7);
              cs[i][r][j] = a.rope[(size_t)pos * half + dim];
            }
          }
      }
      __syncthreads();   // every wave is done with the weight buffers
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            float v = acc[i][j][r];
            const float pv = __shfl_xor(v, 8, 64);
            if (tl.rope) {
              // (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin); lanes ci < 8 hold x1
              const float2 c2 = cs[i][r][j];
              v = v * c2.x + ((ci < 8) ? -pv : pv) * c2.y;
            }
            E[(lr0 + 16 * i + r) * RW + j * 16 + ci] = f32_to_act_bits<F16>(v);
          }
      __syncthreads();
      // piece q: wave-local row q / (2 NB), block (q / 2) % NB, half q % 2
#pragma unroll
      for (int it = 0; it < RB * NB / 2; ++it) {
        const int q = it * 64 + lane;
        const int lr = q / (2 * NB), j = (q >> 1) % NB, h = q & 1;
        const int row = wave * 16 * RB + lr;
        const uint4 v = *reinterpret_cast<const uint4*>(&E[q * 8]);
        const int gb = tl.b0 + j;
        const int col = tl.ocol0 + (gb / hb) * d + (gb % hb) * 8 + h * half;
        if (j < nblk && row < mcnt)
          *reinterpret_cast<uint4*>(out + (size_t)(tl.orow + row) * a.ldo + col) = v;
      }
    } else {
      __syncthreads();   // every wave is done with the weight buffers
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const float gt = acc[i][j][r];
            const float up = __shfl_xor(gt, 8, 64);   // lanes ci < 8: gate, ci >= 8: up
            // silu(g) * u = g / (1 + exp(-g)) * u, reciprocal in hardware
            if (ci < 8)
              E[(lr0 + 16 * i + r) * RW + j * 8 + ci] = f32_to_act_bits<F16>(
                  gt * __builtin_amdgcn_rcpf(1.0f + __expf(-gt)) * up);
          }
      __syncthreads();
      // piece q < 16 RB NB: wave-local row q % (16 RB), block q / (16 RB) (16
      // lanes store the 256 contiguous bytes of one 8-channel group of 16
      // packed rows)
#pragma unroll
      for (int it = 0; it < (RB * NB + 3) / 4; ++it) {
        const int q = it * 64 + lane;
        const int lr = q % (16 * RB), j = q / (16 * RB);
        const int row = wave * 16 * RB + lr;
        if (j < NB) {
          const uint4 v = *reinterpret_cast<const uint4*>(&E[lr * RW + j * 8]);
          if (j < nblk && row < mcnt)
            *reinterpret_cast<uint4*>(out + packed_index((int64_t)tl.orow + row,
                                                         tl.ocol0 + (tl.b0 + j) * 8, a.ldo)) = v;
        }
      }
    }
  } else {
    float* out = EPI == EPI_PARTIAL ? a.partial + (size_t)tl.slice * a.pslice
                                    : static_cast<float*>(a.out);
    float old[RB][4][NB];
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float* orow =
              out + (size_t)(tl.orow + min(rbase + 16 * i + r, mcnt - 1)) * a.ldo + tl.ocol0;
#pragma unroll
          for (int j = 0; j < NB; ++j)
            old[i][r][j] = orow[(tl.b0 + min(j, nblk - 1)) * 16 + ci];
        }
    }
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + 16 * i + r;
        float* orow = out + (size_t)(tl.orow + min(row, mcnt - 1)) * a.ldo + tl.ocol0;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          float v = acc[i][j][r];
          if constexpr (EPI == EPI_RESID) v += old[i][r][j];
          if (j < nblk && row < mcnt) orow[(tl.b0 + j) * 16 + ci] = v;
        }
      }
  }
}

template <int EPI, int NB, bool F16, int NWAVE = 8, bool HILO = false>
hipError_t launch(const MmArgs& a, hipStream_t st) {
  const unsigned grid = (unsigned)((a.ntiles + 7) / 8 * 8);
  gemm_mfma_kernel<EPI, NB, F16, NWAVE, HILO><<<grid, NWAVE * 64, 0, st>>>(a);
  return hipGetLastError();
}

template <int EPI, bool F16, bool HILO = false>
hipError_t by_nb(const MmArgs& a, int32_t nb, hipStream_t st) {
  switch (nb) {
    case 2: return launch<EPI, 2, F16, 8, HILO>(a, st);
    case 3: return launch<EPI, 3, F16, 8, HILO>(a, st);
    case 4: return launch<EPI, 4, F16, 8, HILO>(a, st);
    case 5: return launch<EPI, 5, F16, 8, HILO>(a, st);
    case 6: return launch<EPI, 6, F16, 8, HILO>(a, st);
    case 8: return launch<EPI, 8, F16, 8, HILO>(a, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool F16>
hipError_t dispatch(const MmArgs& a, int32_t epi, int32_t nb, int32_t waves, hipStream_t st) {
  if (waves == 4) {
    // 4-wave tiles: the residual-add output / down projections of 4 blocks
    if (epi == EPI_RESID && nb == 4) return launch<EPI_RESID, 4, F16, 4>(a, st);
    return hipErrorInvalidValue;
  }
  if (waves != 8) return hipErrorInvalidValue;
  if constexpr (!F16) {
    // bf16 products with the activations' low parts (QKV and gate/up)
    if (a.A2 && epi == EPI_QKV) return by_nb<EPI_QKV, false, true>(a, nb, st);
    if (a.A2 && epi == EPI_SWIGLU) return by_nb<EPI_SWIGLU, false, true>(a, nb, st);
  }
  if (a.A2) return hipErrorInvalidValue;   // low parts only for bf16 QKV / gate-up
  switch (epi) {
    case EPI_QKV: return by_nb<EPI_QKV, F16>(a, nb, st);
    case EPI_SWIGLU: return by_nb<EPI_SWIGLU, F16>(a, nb, st);
    case EPI_RESID: return by_nb<EPI_RESID, F16>(a, nb, st);
    case EPI_PARTIAL: return by_nb<EPI_PARTIAL, F16>(a, nb, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_gemm_mfma(const MmArgs& a, int32_t epi, int32_t nb, int32_t waves, bool f16,
                            hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  return f16 ? dispatch<true>(a, epi, nb, waves, st) : dispatch<false>(a, epi, nb, waves, st);
}

}  // namespace svl
