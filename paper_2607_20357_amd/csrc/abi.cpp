// C ABI of libsvl: argument validation (all of it before anything is
// enqueued), workspace layout, one host-to-device copy of the plan per call,
// and the launch sequence of the prefill.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/svl.h"
#include "budget.h"
#include "plan.h"
#include "svl_internal.h"

namespace svl {
namespace {

thread_local std::string g_err;

svl_status fail(svl_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// ------------------------------------------------------------------ timing
struct TimingRec {
  int cls;
  hipEvent_t a, b;
};
struct Timing {
  std::mutex mu;
  bool on = false;
  std::vector<TimingRec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t take() {
    if (!pool.empty()) { hipEvent_t e = pool.back(); pool.pop_back(); return e; }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Timing g_timing;

template <class F>
hipError_t timed(int cls, hipStream_t st, F&& f) {
  if (!g_timing.on) return f();
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    a = g_timing.take();
    b = g_timing.take();
  }
  // an event that fails to record goes back to the pool and the launch runs
  // untimed (timing is a diagnostic; the launch's own status is returned)
  auto give_back = [&] {
    std::lock_guard<std::mutex> lk(g_timing.mu);
    if (a) g_timing.pool.push_back(a);
    if (b) g_timing.pool.push_back(b);
  };
  if (!a || !b || hipEventRecord(a, st) != hipSuccess) {
    give_back();
    return f();
  }
  hipError_t r = f();
  if (hipEventRecord(b, st) != hipSuccess) {
    give_back();
    return r;
  }
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.recs.push_back({cls, a, b});
  return r;
}

enum KClass { K_SELECT = 0, K_GATHER, K_NORM, K_QKV, K_ATTN, K_O, K_GU, K_DOWN, K_ROPE, K_FINISH,
              K_KV_APPEND, K_CTRL };

// ------------------------------------------------------------------ validation
svl_status check_config(const svl_config* c, bool for_kernels = true) {
  if (!c) return fail(SVL_E_NULL, "config is NULL");
  if (c->dtype != SVL_F32 && c->dtype != SVL_BF16) return fail(SVL_E_DTYPE, "unknown dtype %d", c->dtype);
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->d_ffn <= 0 || c->n_groups <= 0)
    return fail(SVL_E_SHAPE, "every size in the config must be positive");
  if (c->n_heads % c->n_kv_heads) return fail(SVL_E_SHAPE, "n_heads %% n_kv_heads != 0");
  if (c->head_dim % 2) return fail(SVL_E_SHAPE, "head_dim must be even (RoPE pairs)");
  if (c->d_ffn % c->n_groups) return fail(SVL_E_SHAPE, "d_ffn %% n_groups != 0");
  if (!(c->rms_eps >= 0.f)) return fail(SVL_E_VALUE, "rms_eps must be >= 0");
  if (!(c->rope_theta > 0.f)) return fail(SVL_E_VALUE, "rope_theta must be > 0");
  if (c->compute != SVL_COMPUTE_F16 && c->compute != SVL_COMPUTE_BF16)
    return fail(SVL_E_DTYPE, "unknown compute type %d", c->compute);
  if (!for_kernels) return SVL_OK;
  if (c->dtype == SVL_BF16) {
    if (c->d_model % 64) return fail(SVL_E_SHAPE, "bf16 path: d_model %% 64 != 0");
    if (c->head_dim != 64 && c->head_dim != 128)
      return fail(SVL_E_SHAPE, "bf16 path: head_dim must be 64 or 128");
    if ((c->d_ffn / c->n_groups) % 64) return fail(SVL_E_SHAPE, "bf16 path: d_ffn/n_groups %% 64 != 0");
    if (c->d_model > 65536 || c->d_ffn > 65536 || c->n_heads * c->head_dim > 65536)
      return fail(SVL_E_SHAPE, "bf16 path: reduction dimensions above 65536");
    // the GEMM kernels address a weight matrix with 32-bit byte offsets below 2^31
    const int64_t D = c->d_model, F = c->d_ffn, Ad = (int64_t)c->n_heads * c->head_dim;
    if (F * D * 2 >= (int64_t(1) << 31) || Ad * D * 2 >= (int64_t(1) << 31))
      return fail(SVL_E_SHAPE, "bf16 path: a weight matrix of 2 GiB or more");
  } else {
    if (c->d_model % 4) return fail(SVL_E_SHAPE, "f32 path: d_model %% 4 != 0");
    if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
      return fail(SVL_E_SHAPE, "f32 path: head_dim must be 32, 64 or 128");
  }
  return SVL_OK;
}

svl_status check_mask(const uint8_t* m, int64_t n, const char* what) {
  for (int64_t i = 0; i < n; ++i)
    if (m[i] > 1) return fail(SVL_E_VALUE, "%s[%lld] = %u is not 0 or 1", what, (long long)i, m[i]);
  return SVL_OK;
}

// ------------------------------------------------------------------ workspace
struct WsLayout {
  int64_t plan, rope, partial, xn, xn_lo, qkv, attn_out, h, total;
  int64_t partial_slice;   // floats per split-K slice of the output / down projections (R x d_model)
  int64_t prows;           // padded activation rows
};

// Activation buffers use the padded row space (16-row blocks per sample on
// the 16-bit MFMA path); the partial region holds the float32 split-K slices.
// pos_rows: RoPE table rows (positions) when they exceed R (decode: max_len).
// Decode (pos_rows > 0) never splits K, so its layout has no partial region.
// The status word: the last four bytes of the caller's workspace buffer
// (inside the 256 bytes every layout reserves at its end, or past the
// layout when the buffer is larger).
uint32_t* status_word(void* ws, size_t ws_bytes) {
  return reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(ws) + ((ws_bytes & ~size_t(3)) - 4));
}

// bf16 activations (bf16 storage, SVL_COMPUTE_BF16) carry the normed rows
// as two bf16 terms, hi = bf16(x) and lo = bf16(x - hi), into the QKV and
// gate/up products (both multiplied by bf16 MFMA, summed in float32).
bool lo_parts(const svl_config& c) {
  return c.dtype == SVL_BF16 && c.compute == SVL_COMPUTE_BF16;
}

WsLayout ws_layout(const svl_config& c, int32_t B, int32_t R, int32_t pos_rows = 0) {
  const int64_t es = c.dtype == SVL_BF16 ? 2 : 4;
  const int64_t prow = std::max<int64_t>(padded_rows_bound(c, B, R), 16);
  WsLayout L{};
  int64_t off = 0;
  auto take = [&](int64_t bytes) {
    int64_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.plan = take(plan_bytes_bound(c, B, R, c.n_layers));
  L.rope = take(std::max<int64_t>(std::max(R, pos_rows), 1) * (c.head_dim / 2) * 8);
  L.partial = take(pos_rows > 0 ? 0 : partial_floats_bound(c, B, R) * 4);
  L.partial_slice = (int64_t)R * c.d_model;
  L.prows = prow;
  L.xn = take(prow * c.d_model * es);
  // bf16 activations: the normed rows' low bf16 parts, for the QKV and
  // gate/up products
  L.xn_lo = take(lo_parts(c) ? prow * c.d_model * 2 : 0);
  L.qkv = take(prow * (int64_t)(c.n_heads + 2 * c.n_kv_heads) * c.head_dim * es);
  L.attn_out = take(prow * (int64_t)c.n_heads * c.head_dim * es);
  L.h = take(prow * (int64_t)c.d_ffn * es);
  take(256);   // the last bytes of the buffer hold the call's status word (svl_workspace_status)
  L.total = off;
  return L;
}

// ------------------------------------------------------------------ execution
struct Exec {
  const svl_config& c;
  hipStream_t st;
  uint8_t* ws;
  WsLayout L;
  const Plan& plan;
  float* resid;
  // KV cache (decode stage): [layers][batch][KV][2][max_len][d]; nullptr: none
  uint8_t* cache = nullptr;
  int32_t max_len = 0;
  int32_t batch = 0;
  bool decode = false;   // one new row per sample: attention over the cache

  template <class T>
  const T* at(int64_t off) const { return reinterpret_cast<const T*>(ws + L.plan + off); }

  hipError_t gemm(const GemmLaunch& g, const KChunk* chunks, const void* A, int lda, const void* W0,
                  const void* W1, const void* W2, int ldw, int nb1, int nb2, void* out, int ldo,
                  int epi, int cls) const {
    if (g.ntiles == 0) return hipSuccess;
    GemmArgs a{};
    a.groups = at<GemmGroup>(g.groups_off);
    a.ngroups = g.ngroups;
    a.ntiles = g.ntiles;
    a.chunks = chunks;
    a.A = A; a.lda = lda;
    a.W0 = W0; a.W1 = W1; a.W2 = W2; a.ldw = ldw; a.nb1 = nb1; a.nb2 = nb2;
    a.out = out; a.ldo = ldo;
    a.rope = reinterpret_cast<const float2*>(ws + L.rope);
    a.head_dim = c.head_dim;
    a.rope_cols = (c.n_heads + c.n_kv_heads) * c.head_dim;
    a.partial = reinterpret_cast<float*>(ws + L.partial);
    a.pslice = L.partial_slice;
    return timed(cls, st, [&] { return launch_gemm_f32(a, epi, st); });
  }

  // 16-bit MFMA GEMM over the launch's tile table.  W holds up to three
  // weight matrices with their row counts.
  hipError_t mm(const GemmLaunch& g, const KChunk* chunks, const void* A, int lda,
                const void* const (&W)[3], const int32_t (&w_rows)[3], int ldw, void* out, int ldo,
                int epi, int cls) const {
    if (g.ntiles == 0) return hipSuccess;
    MmArgs a{};
    a.groups = at<MmGroup>(g.groups_off);
    a.tiles = at<MmTile>(g.tiles_off);
    a.ntiles = g.ntiles;
    a.chunks = chunks;
    a.A = A; a.lda = lda;
    // the normed rows' low parts (QKV and gate/up products of bf16 activations)
    if (!decode && lo_parts(c) && A == ws + L.xn && (epi == EPI_QKV || epi == EPI_SWIGLU))
      a.A2 = ws + L.xn_lo;
    for (int i = 0; i < 3; ++i) { a.W[i] = W[i]; a.w_rows[i] = w_rows[i]; }
    a.ldw = ldw;
    a.out = out; a.ldo = ldo;
    a.rope = reinterpret_cast<const float2*>(ws + L.rope);
    a.head_dim = c.head_dim;
    a.partial = reinterpret_cast<float*>(ws + L.partial);
    a.rowpos = at<int32_t>(plan.rowpos_off);
    const bool f16 = c.compute == SVL_COMPUTE_F16;
    if (decode) {
      // one row per sample: row-vector products over the groups' blocks, or
      // over the shared segments (a batch: each weight block read once for
      // all samples using it)
      a.ngroups = g.ngroups;
      a.nblocks = g.nblocks;
      if (g.nsegs > 0) {
        a.segs = at<DecSeg>(g.segs_off);
        a.nsegs = g.nsegs;
        a.uses = at<DecUse>(g.uses_off);
        a.cmasks = at<int32_t>(g.cmasks_off);
        a.max_uses = g.max_uses;
        return timed(cls, st, [&] { return launch_gemv_shared(a, epi, f16, st); });
      }
      return timed(cls, st, [&] { return launch_gemv(a, epi, f16, st); });
    }
    const bool paired = epi == EPI_QKV || epi == EPI_SWIGLU;
    if (paired && g.nsplit > 1) {
      // split pieces: float32 slices [nsplit][padded rows][pld], then the finish
      a.split = g.nsplit;
      a.pld = epi == EPI_QKV ? ldo : 2 * c.d_ffn;
      a.pslice = plan.padded_rows * (int64_t)a.pld;
    } else {
      a.split = 1;
      a.pld = ldo;
      a.pslice = L.partial_slice;
    }
    hipError_t e = timed(cls, st, [&] { return launch_gemm_mfma(a, epi, g.nb, g.waves, f16, st); });
    if (e != hipSuccess || !(paired && g.nsplit > 1)) return e;
    FinishArgs f{};
    f.groups = a.groups;
    f.ngroups = g.ngroups;
    f.nitems = g.nitems;
    f.partial = a.partial;
    f.pslice = a.pslice;
    f.pld = a.pld;
    f.nsplit = g.nsplit;
    f.out = out;
    f.ldo = ldo;
    f.rope = a.rope;
    f.head_dim = c.head_dim;
    return timed(K_FINISH, st, [&] { return launch_finish(f, epi, f16, st); });
  }

  hipError_t norm(const NormLaunch& n, const void* gain) const {
    if (n.nrows == 0) return hipSuccess;
    NormArgs a{};
    a.segs = at<NormSeg>(n.segs_off);
    a.nsegs = n.nsegs;
    const NormSeg* hs = reinterpret_cast<const NormSeg*>(plan.image.data() + n.segs_off);
    for (int32_t i = 0; i < n.nsegs; ++i)   // normed rows need the gain
      if ((hs[i].flags & NORM_WRITE_OUT) && gain == nullptr) return hipErrorInvalidValue;
    if (n.nsegs <= NORM_INLINE_SEGS) std::memcpy(a.inl, hs, (size_t)n.nsegs * sizeof(NormSeg));
    a.nrows = n.nrows;
    a.ngroups8 = n.ngroups8;
    a.rows8 = n.rows8 ? 1 : 0;
    a.rowmajor = decode ? 1 : 0;   // decode: row-vector products read row-major rows
    a.x = resid;
    a.partial = reinterpret_cast<const float*>(ws + L.partial);
    a.nsplit = n.nsplit;
    a.pslice = L.partial_slice;
    a.gain = gain;
    a.out = ws + L.xn;
    a.out2 = !decode && lo_parts(c) ? ws + L.xn_lo : nullptr;
    a.D = c.d_model;
    a.eps = c.rms_eps;
    const int out_kind = c.dtype != SVL_BF16 ? 0 : (c.compute == SVL_COMPUTE_F16 ? 2 : 1);
    return timed(K_NORM, st, [&] { return launch_resid_norm(a, out_kind, st); });
  }

  // Output / down projection: straight into the residual, or split-K
  // pieces into the partial slices the next residual-finish launch adds.
  static int resid_epi(const GemmLaunch& g) { return g.nsplit > 1 ? EPI_PARTIAL : EPI_RESID; }

  hipError_t layer(const LayerPlan& P, const svl_layer_weights& w, int32_t l = 0) const {
    const int A = c.n_heads, KV = c.n_kv_heads, d = c.head_dim, D = c.d_model, F = c.d_ffn;
    const int qkv_w = (A + 2 * KV) * d;
    const bool mfma = c.dtype == SVL_BF16;
    const KChunk* chunks = at<KChunk>(P.chunks_off);
    hipError_t e = hipSuccess;
    if ((e = norm(P.norm_attn, w.attn_norm)) != hipSuccess) return e;
    if (P.qkv.ntiles > 0) {
      if (mfma) {
        const void* const W[3] = {w.wq, w.wk, w.wv};
        const int32_t rows[3] = {A * d, KV * d, KV * d};
        e = mm(P.qkv, chunks, ws + L.xn, D, W, rows, D, ws + L.qkv, qkv_w, EPI_QKV, K_QKV);
      } else {
        e = gemm(P.qkv, chunks, ws + L.xn, D, w.wq, w.wk, w.wv, D, A * d, (A + KV) * d,
                 ws + L.qkv, qkv_w, EPI_STORE, K_QKV);
      }
      if (e != hipSuccess) return e;
      AttnArgs a{};
      a.groups = at<AttnGroup>(P.attn.groups_off);
      a.ngroups = P.attn.ngroups;
      a.ntiles = P.attn.ntiles;
      a.bq = P.attn.bq;
      a.head_table = at<int32_t>(P.attn.heads_off);
      a.qkv = ws + L.qkv;
      a.ldq = qkv_w;
      a.n_heads = A;
      a.n_kv_heads = KV;
      a.out = ws + L.attn_out;
      a.ldo = A * d;
      a.rope = reinterpret_cast<const float2*>(ws + L.rope);
      a.scale = 1.0f / std::sqrt((float)d);
      // active K/V heads per group: the cache append and the grouped-K/V
      // prefill attention read them
      a.kvhead_table = at<int32_t>(P.attn.kvheads_off);
      a.max_kv_cnt = P.attn.max_kv_cnt;
      if (cache) {
        a.cache = cache + (size_t)l * batch * KV * 2 * (size_t)max_len * d * 2;
        a.max_len = max_len;
        // prefill: this call's K / V rows into the cache (decode attention
        // appends its one row itself)
        if (!decode) {
          e = timed(K_KV_APPEND, st, [&] { return launch_kv_append(a, d, st); });
          if (e != hipSuccess) return e;
        }
      }
      e = timed(K_ATTN, st, [&] {
        if (decode) return launch_attn_decode(a, d, c.compute == SVL_COMPUTE_F16, st);
        return mfma ? launch_attn_mfma(a, d, c.compute == SVL_COMPUTE_F16, st)
                    : launch_attn_f32(a, d, st);
      });
      if (e != hipSuccess) return e;
      if (mfma) {
        const void* const W[3] = {w.wo, nullptr, nullptr};
        const int32_t rows[3] = {D, 0, 0};
        e = mm(P.o, chunks, ws + L.attn_out, A * d, W, rows, A * d, resid, D, resid_epi(P.o), K_O);
      } else {
        e = gemm(P.o, chunks, ws + L.attn_out, A * d, w.wo, nullptr, nullptr, A * d, 0, 0, resid,
                 D, resid_epi(P.o), K_O);
      }
      if (e != hipSuccess) return e;
    }
    if ((e = norm(P.norm_ffn, w.ffn_norm)) != hipSuccess) return e;
    if (P.gu.ntiles > 0) {
      if (mfma) {
        const void* const Wg[3] = {w.w_gate, w.w_up, nullptr};
        const int32_t rg[3] = {F, F, 0};
        if ((e = mm(P.gu, chunks, ws + L.xn, D, Wg, rg, D, ws + L.h, F, EPI_SWIGLU, K_GU)) !=
            hipSuccess)
          return e;
        const void* const Wd[3] = {w.w_down, nullptr, nullptr};
        const int32_t rd[3] = {D, 0, 0};
        e = mm(P.down, chunks, ws + L.h, F, Wd, rd, F, resid, D, resid_epi(P.down), K_DOWN);
      } else {
        if ((e = gemm(P.gu, chunks, ws + L.xn, D, w.w_gate, w.w_up, nullptr, D, 0, 0, ws + L.h, F,
                      EPI_SWIGLU, K_GU)) != hipSuccess)
          return e;
        e = gemm(P.down, chunks, ws + L.h, F, w.w_down, nullptr, nullptr, F, 0, 0, resid, D,
                 resid_epi(P.down), K_DOWN);
      }
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
};

thread_local Plan t_plan;

svl_status hip_fail(hipError_t e, const char* where) {
  return fail(SVL_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

// Plan uploads go through two pinned host buffers per thread, used in turn:
// the image is copied into one (after the copy that last read it has
// completed, which its event tells) and the stream copies it to the
// workspace asynchronously, so the host does not stage pageable memory
// while the GPU waits.  The buffers and events live until the process ends
// (they are never released, so no teardown runs after the HIP runtime's).
struct PinnedRing {
  uint8_t* buf[2] = {nullptr, nullptr};
  size_t cap[2] = {0, 0};
  hipEvent_t done[2] = {nullptr, nullptr};
  bool pending[2] = {false, false};
  int next = 0;
  int device = -1;   // the events belong to this device
};
thread_local PinnedRing t_ring;

hipError_t upload_plan(uint8_t* dst, const uint8_t* src, size_t n, hipStream_t st) {
  PinnedRing& r = t_ring;
  hipError_t e;
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if (dev != r.device) {
    // another device: let the pending copies finish, then start fresh events
    // (the old ones are left to the process end, like the buffers)
    for (int j = 0; j < 2; ++j) {
      if (r.pending[j] && (e = hipEventSynchronize(r.done[j])) != hipSuccess) return e;
      r.pending[j] = false;
      r.done[j] = nullptr;
    }
    r.device = dev;
  }
  const int i = r.next;
  r.next ^= 1;
  if (!r.done[i] && (e = hipEventCreateWithFlags(&r.done[i], hipEventDisableTiming)) != hipSuccess)
    return e;
  if (r.pending[i] && (e = hipEventSynchronize(r.done[i])) != hipSuccess) return e;
  r.pending[i] = false;
  if (r.cap[i] < n) {
    if (r.buf[i] && (e = hipHostFree(r.buf[i])) != hipSuccess) return e;
    r.buf[i] = nullptr;
    r.cap[i] = 0;
    const size_t cap = n + n / 2 + 4096;
    void* p = nullptr;
    if ((e = hipHostMalloc(&p, cap, hipHostMallocDefault)) != hipSuccess) return e;
    r.buf[i] = static_cast<uint8_t*>(p);
    r.cap[i] = cap;
  }
  std::memcpy(r.buf[i], src, n);
  if ((e = hipMemcpyAsync(dst, r.buf[i], n, hipMemcpyHostToDevice, st)) != hipSuccess) return e;
  if ((e = hipEventRecord(r.done[i], st)) != hipSuccess) return e;
  r.pending[i] = true;
  return hipSuccess;
}

// Copies the plan image and builds the RoPE table.  pageable: copy straight
// from the plan's host memory (the allocation-free entry point; a copy from
// pageable memory has consumed its source when the call returns) instead of
// through the pinned buffers, which are allocated on first use.
svl_status stage(const Exec& ex, bool need_layers, bool pageable = false) {
  if ((int64_t)ex.plan.image.size() > ex.L.rope - ex.L.plan)
    return fail(SVL_E_SHAPE, "internal: plan image exceeds its workspace region");
  hipError_t e =
      pageable ? hipMemcpyAsync(ex.ws + ex.L.plan, ex.plan.image.data(), ex.plan.image.size(),
                                hipMemcpyHostToDevice, ex.st)
               : upload_plan(ex.ws + ex.L.plan, ex.plan.image.data(), ex.plan.image.size(), ex.st);
  if (e != hipSuccess) return hip_fail(e, "plan upload");
  if (need_layers) {
    e = timed(K_ROPE, ex.st, [&] {
      return launch_rope_table(reinterpret_cast<float2*>(ex.ws + ex.L.rope), ex.plan.max_pos,
                               ex.c.head_dim, ex.c.rope_theta, ex.st);
    });
    if (e != hipSuccess) return hip_fail(e, "rope table");
  }
  return SVL_OK;
}

svl_status check_batch(const svl_config& c, const svl_batch* b) {
  if (!b) return fail(SVL_E_NULL, "batch is NULL");
  if (b->batch <= 0) return fail(SVL_E_SHAPE, "batch must be positive");
  if (b->n_vision < 0 || b->n_text < 0) return fail(SVL_E_SHAPE, "negative token counts");
  if (!b->keep) return fail(SVL_E_NULL, "keep is NULL");
  int64_t total = 0;
  for (int32_t i = 0; i < b->batch; ++i) {
    if (b->keep[i] < 0 || b->keep[i] > b->n_vision)
      return fail(SVL_E_VALUE, "keep[%d] = %d outside [0, %d]", i, b->keep[i], b->n_vision);
    total += b->keep[i] + b->n_text;
  }
  if (total > INT32_MAX) return fail(SVL_E_SHAPE, "too many packed rows");
  (void)c;
  return SVL_OK;
}

svl_status check_ws(const svl_config& c, int32_t B, int32_t R, void* ws, size_t ws_bytes) {
  if (!ws) return fail(SVL_E_NULL, "workspace is NULL");
  if (!aligned16(ws)) return fail(SVL_E_ALIGN, "workspace not 16-byte aligned");
  const WsLayout L = ws_layout(c, B, R);
  if ((int64_t)ws_bytes < L.total)
    return fail(SVL_E_WORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)L.total);
  return SVL_OK;
}

// Data pointers: scores, vision and kept_idx are needed when there are vision
// tokens, text when there are text tokens, resid when there are packed rows.
svl_status check_data(const svl_batch& b, int32_t R, const void* scores, const void* vision,
                      const void* text, const void* kept_idx, const void* resid) {
  if (b.n_vision > 0 && (!scores || !vision || !kept_idx))
    return fail(SVL_E_NULL, "scores, vision and kept_idx are required when n_vision > 0");
  if (b.n_text > 0 && !text) return fail(SVL_E_NULL, "text is required when n_text > 0");
  if (R > 0 && !resid) return fail(SVL_E_NULL, "resid is required when there are packed rows");
  for (const void* p : {scores, vision, text, kept_idx, resid})
    if (p && !aligned16(p)) return fail(SVL_E_ALIGN, "device pointers must be 16-byte aligned");
  return SVL_OK;
}

svl_status select_and_gather(const Exec& ex, const svl_batch& b, const float* scores,
                             const void* vision, const void* text, int32_t* kept_idx, int32_t R) {
  const int32_t* keep_dev = ex.at<int32_t>(ex.plan.keep_off);
  const int32_t* cu_dev = ex.at<int32_t>(ex.plan.cu_off);
  hipError_t e = timed(K_SELECT, ex.st, [&] {
    return launch_select(scores, b.batch, b.n_vision, keep_dev, kept_idx, ex.st);
  });
  if (e != hipSuccess) return hip_fail(e, "select");
  e = timed(K_GATHER, ex.st, [&] {
    return launch_gather(kept_idx, keep_dev, cu_dev, b.batch, b.n_vision, b.n_text, ex.c.d_model, R,
                         vision, text, ex.c.dtype, ex.resid, ex.st);
  });
  if (e != hipSuccess) return hip_fail(e, "gather");
  return SVL_OK;
}

void closed_form(const svl_config& c, int64_t S, const uint8_t* hm, const uint8_t* fm, svl_flops* f) {
  const int64_t D = c.d_model, d = c.head_dim, A = c.n_heads, KV = c.n_kv_heads, G = c.n_groups;
  const int64_t rep = A / KV;
  int64_t H = 0, K = 0, C = 0;
  for (int64_t h = 0; h < A; ++h) H += hm[h] ? 1 : 0;
  for (int64_t g = 0; g < KV; ++g) {
    bool on = false;
    for (int64_t h = g * rep; h < (g + 1) * rep; ++h) on = on || hm[h];
    K += on ? 1 : 0;
  }
  if (fm) { for (int64_t j = 0; j < G; ++j) C += fm[j] ? c.d_ffn / G : 0; } else { C = c.d_ffn; }
  f->q += 2 * S * D * d * H;
  f->kv += 4 * S * D * d * K;
  f->o += 2 * S * H * d * D;
  f->attn += 2 * H * d * S * (S + 1);
  f->ffn += 6 * S * D * C;
}

}  // namespace

// Error reporting and the config check, shared with the other C-ABI sources.
svl_status set_error(svl_status st, const char* msg) {
  g_err = msg;
  return st;
}
svl_status validate_config(const svl_config* c) { return check_config(c); }

}  // namespace svl

using namespace svl;

extern "C" {

const char* svl_last_error(void) { return g_err.c_str(); }

int32_t svl_abi_version(void) { return SVL_ABI_VERSION; }

size_t svl_workspace_bytes(const svl_config* cfg, int32_t batch, int32_t total_rows) {
  if (check_config(cfg) != SVL_OK || batch <= 0 || total_rows < 0) return 0;
  return (size_t)ws_layout(*cfg, batch, total_rows).total;
}

svl_status svl_count_flops(const svl_config* cfg, int32_t batch, const int32_t* seqlens,
                           const uint8_t* layer_mask, const uint8_t* head_mask,
                           const uint8_t* ffn_mask, svl_flops* out) {
  svl_status s = check_config(cfg, false);
  if (s != SVL_OK) return s;
  if (batch <= 0) return fail(SVL_E_SHAPE, "batch must be positive");
  if (!seqlens || !layer_mask || !head_mask || !out) return fail(SVL_E_NULL, "NULL argument");
  const int64_t L = cfg->n_layers, A = cfg->n_heads, G = cfg->n_groups;
  if ((s = check_mask(layer_mask, batch * L, "layer_mask")) != SVL_OK) return s;
  if ((s = check_mask(head_mask, batch * L * A, "head_mask")) != SVL_OK) return s;
  if (ffn_mask && (s = check_mask(ffn_mask, batch * L * G, "ffn_mask")) != SVL_OK) return s;
  svl_flops f{};
  for (int64_t b = 0; b < batch; ++b) {
    if (seqlens[b] < 0) return fail(SVL_E_VALUE, "negative sequence length");
    for (int64_t l = 0; l < L; ++l)
      if (layer_mask[b * L + l])
        closed_form(*cfg, seqlens[b], head_mask + (b * L + l) * A,
                    ffn_mask ? ffn_mask + (b * L + l) * G : nullptr, &f);
  }
  f.total = f.q + f.kv + f.o + f.attn + f.ffn;
  *out = f;
  return SVL_OK;
}

svl_status svl_select_tokens(const svl_config* cfg, const svl_batch* batch, const float* scores,
                             const void* vision, const void* text, int32_t* kept_idx, float* resid,
                             int32_t* cu_seqlens, void* ws, size_t ws_bytes, void* stream) {
  svl_status s = check_config(cfg);
  if (s != SVL_OK) return s;
  if ((s = check_batch(*cfg, batch)) != SVL_OK) return s;
  const int32_t B = batch->batch;
  std::vector<int32_t> seq(B);
  int32_t R = 0;
  for (int32_t b = 0; b < B; ++b) { seq[b] = batch->keep[b] + batch->n_text; R += seq[b]; }
  if (!cu_seqlens) return fail(SVL_E_NULL, "cu_seqlens is NULL");
  if ((s = check_data(*batch, R, scores, vision, text, kept_idx, resid)) != SVL_OK) return s;
  if ((s = check_ws(*cfg, B, R, ws, ws_bytes)) != SVL_OK) return s;
  std::string err;
  if (!build_plan(*cfg, B, batch->keep, seq.data(), 0, nullptr, &t_plan, &err))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  cu_seqlens[0] = 0;
  for (int32_t b = 0; b < B; ++b) cu_seqlens[b + 1] = cu_seqlens[b] + seq[b];
  Exec ex{*cfg, (hipStream_t)stream, static_cast<uint8_t*>(ws), ws_layout(*cfg, B, R), t_plan, resid};
  if ((s = stage(ex, false)) != SVL_OK) return s;
  return select_and_gather(ex, *batch, scores, vision, text, kept_idx, R);
}

svl_status svl_layer_forward(const svl_config* cfg, int32_t layer, const svl_layer_weights* w,
                             int32_t batch, const int32_t* cu_seqlens, const uint8_t* layer_on,
                             const uint8_t* head_mask, const uint8_t* ffn_mask, float* resid,
                             void* ws, size_t ws_bytes, void* stream) {
  svl_status s = check_config(cfg);
  if (s != SVL_OK) return s;
  if (layer < 0 || layer >= cfg->n_layers) return fail(SVL_E_VALUE, "layer index out of range");
  if (batch <= 0) return fail(SVL_E_SHAPE, "batch must be positive");
  if (!w || !cu_seqlens || !layer_on || !head_mask || !resid) return fail(SVL_E_NULL, "NULL argument");
  const void* wp[9] = {w->attn_norm, w->wq, w->wk, w->wv, w->wo, w->ffn_norm, w->w_gate, w->w_up, w->w_down};
  for (const void* p : wp) {
    if (!p) return fail(SVL_E_NULL, "NULL weight pointer");
    if (!aligned16(p)) return fail(SVL_E_ALIGN, "weight pointers must be 16-byte aligned");
  }
  if (!aligned16(resid)) return fail(SVL_E_ALIGN, "resid must be 16-byte aligned");
  if (cu_seqlens[0] != 0) return fail(SVL_E_VALUE, "cu_seqlens[0] must be 0");
  std::vector<int32_t> seq(batch);
  for (int32_t b = 0; b < batch; ++b) {
    seq[b] = cu_seqlens[b + 1] - cu_seqlens[b];
    if (seq[b] < 0) return fail(SVL_E_VALUE, "cu_seqlens must be non-decreasing");
  }
  const int32_t R = cu_seqlens[batch];
  if ((s = check_mask(layer_on, batch, "layer_on")) != SVL_OK) return s;
  if ((s = check_mask(head_mask, (int64_t)batch * cfg->n_heads, "head_mask")) != SVL_OK) return s;
  if (ffn_mask && (s = check_mask(ffn_mask, (int64_t)batch * cfg->n_groups, "ffn_mask")) != SVL_OK)
    return s;
  if ((s = check_ws(*cfg, batch, R, ws, ws_bytes)) != SVL_OK) return s;
  LayerMasks m{layer_on, head_mask, cfg->n_heads, ffn_mask, cfg->n_groups};
  std::string err;
  if (!build_plan(*cfg, batch, nullptr, seq.data(), 1, &m, &t_plan, &err))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  Exec ex{*cfg, (hipStream_t)stream, static_cast<uint8_t*>(ws), ws_layout(*cfg, batch, R), t_plan, resid};
  if ((s = stage(ex, true)) != SVL_OK) return s;
  hipError_t e = ex.layer(t_plan.layers[0], *w);
  if (e == hipSuccess) e = ex.norm(t_plan.final_norm, nullptr);
  if (e != hipSuccess) return hip_fail(e, "layer launch");
  return SVL_OK;
}

// Host masks [B][L][...] -> per-layer LayerMasks (lon: the transposed layer mask).
static void layer_masks(const svl_config& c, int32_t B, const uint8_t* layer_mask,
                        const uint8_t* head_mask, const uint8_t* ffn_mask,
                        std::vector<LayerMasks>& masks, std::vector<uint8_t>& lon) {
  const int32_t L = c.n_layers, A = c.n_heads, G = c.n_groups;
  masks.assign(L, LayerMasks{});
  lon.assign((size_t)L * B, 0);
  for (int32_t l = 0; l < L; ++l) {
    // row b of layer l starts at (b*L + l) * width
    masks[l].head_mask = head_mask + (int64_t)l * A;
    masks[l].head_stride = (int64_t)L * A;
    masks[l].ffn_mask = ffn_mask ? ffn_mask + (int64_t)l * G : nullptr;
    masks[l].ffn_stride = (int64_t)L * G;
    for (int32_t b = 0; b < B; ++b) lon[(size_t)l * B + b] = layer_mask[(int64_t)b * L + l];
    masks[l].layer_on = lon.data() + (size_t)l * B;
  }
}

static svl_status check_layers(const svl_config& c, const svl_layer_weights* layers) {
  if (!layers) return fail(SVL_E_NULL, "layers is NULL");
  for (int32_t l = 0; l < c.n_layers; ++l) {
    const svl_layer_weights& w = layers[l];
    const void* wp[9] = {w.attn_norm, w.wq, w.wk, w.wv, w.wo, w.ffn_norm, w.w_gate, w.w_up, w.w_down};
    for (const void* p : wp) {
      if (!p) return fail(SVL_E_NULL, "NULL weight pointer in layer %d", l);
      if (!aligned16(p)) return fail(SVL_E_ALIGN, "weight pointer of layer %d not 16-byte aligned", l);
    }
  }
  return SVL_OK;
}

// The prefill, optionally writing every layer's K / V rows into a cache.
static svl_status prefill_impl(const svl_config* cfg, const svl_layer_weights* layers,
                               const svl_batch* batch, const float* scores, const void* vision,
                               const void* text, const uint8_t* layer_mask,
                               const uint8_t* head_mask, const uint8_t* ffn_mask,
                               int32_t* kept_idx, float* resid, int32_t* cu_seqlens,
                               svl_flops* flops, void* ws, size_t ws_bytes, void* stream,
                               void* cache, int32_t max_len) {
  svl_status s = check_config(cfg);
  if (s != SVL_OK) return s;
  if ((s = check_batch(*cfg, batch)) != SVL_OK) return s;
  if (!layer_mask || !head_mask || !cu_seqlens) return fail(SVL_E_NULL, "NULL argument");
  const int32_t B = batch->batch, L = cfg->n_layers, A = cfg->n_heads, G = cfg->n_groups;
  std::vector<int32_t> seq(B);
  int32_t R = 0;
  for (int32_t b = 0; b < B; ++b) { seq[b] = batch->keep[b] + batch->n_text; R += seq[b]; }
  if ((s = check_data(*batch, R, scores, vision, text, kept_idx, resid)) != SVL_OK) return s;
  if ((s = check_layers(*cfg, layers)) != SVL_OK) return s;
  if ((s = check_mask(layer_mask, (int64_t)B * L, "layer_mask")) != SVL_OK) return s;
  if ((s = check_mask(head_mask, (int64_t)B * L * A, "head_mask")) != SVL_OK) return s;
  if (ffn_mask && (s = check_mask(ffn_mask, (int64_t)B * L * G, "ffn_mask")) != SVL_OK) return s;
  if (cache) {
    if (cfg->dtype != SVL_BF16) return fail(SVL_E_DTYPE, "the KV cache is on the 16-bit path only");
    if (!aligned16(cache)) return fail(SVL_E_ALIGN, "kv_cache not 16-byte aligned");
    if (max_len <= 0 || max_len > 32768) return fail(SVL_E_SHAPE, "max_len outside [1, 32768]");
    for (int32_t b = 0; b < B; ++b)
      if (seq[b] > max_len) return fail(SVL_E_SHAPE, "sample %d has %d rows > max_len %d", b, seq[b], max_len);
  }
  if ((s = check_ws(*cfg, B, R, ws, ws_bytes)) != SVL_OK) return s;
  std::vector<LayerMasks> masks;
  std::vector<uint8_t> lon;
  layer_masks(*cfg, B, layer_mask, head_mask, ffn_mask, masks, lon);
  std::string err;
  if (!build_plan(*cfg, B, batch->keep, seq.data(), L, masks.data(), &t_plan, &err))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  cu_seqlens[0] = 0;
  for (int32_t b = 0; b < B; ++b) cu_seqlens[b + 1] = cu_seqlens[b] + seq[b];
  if (flops) {
    svl_status fs = svl_count_flops(cfg, B, seq.data(), layer_mask, head_mask, ffn_mask, flops);
    if (fs != SVL_OK) return fs;
  }
  Exec ex{*cfg, (hipStream_t)stream, static_cast<uint8_t*>(ws), ws_layout(*cfg, B, R), t_plan, resid};
  ex.cache = static_cast<uint8_t*>(cache);
  ex.max_len = max_len;
  ex.batch = B;
  if ((s = stage(ex, true)) != SVL_OK) return s;
  if ((s = select_and_gather(ex, *batch, scores, vision, text, kept_idx, R)) != SVL_OK) return s;
  for (int32_t l = 0; l < L; ++l) {
    hipError_t e = ex.layer(t_plan.layers[l], layers[l], l);
    if (e != hipSuccess) return hip_fail(e, "layer launch");
  }
  hipError_t e = ex.norm(t_plan.final_norm, nullptr);
  if (e != hipSuccess) return hip_fail(e, "final residual launch");
  // the status word: cleared, then set if an output value is inf or NaN
  uint32_t* status = status_word(ws, ws_bytes);
  if ((e = launch_fill_i32(reinterpret_cast<int32_t*>(status), 0, 1, ex.st)) != hipSuccess)
    return hip_fail(e, "status clear");
  if ((e = launch_nonfinite(resid, (int64_t)R * cfg->d_model, status, ex.st)) != hipSuccess)
    return hip_fail(e, "status scan");
  return SVL_OK;
}

svl_status svl_prefill(const svl_config* cfg, const svl_layer_weights* layers, const svl_batch* batch,
                       const float* scores, const void* vision, const void* text,
                       const uint8_t* layer_mask, const uint8_t* head_mask, const uint8_t* ffn_mask,
                       int32_t* kept_idx, float* resid, int32_t* cu_seqlens, svl_flops* flops,
                       void* ws, size_t ws_bytes, void* stream) {
  return prefill_impl(cfg, layers, batch, scores, vision, text, layer_mask, head_mask, ffn_mask,
                      kept_idx, resid, cu_seqlens, flops, ws, ws_bytes, stream, nullptr, 0);
}

svl_status svl_prefill_cache(const svl_config* cfg, const svl_layer_weights* layers,
                             const svl_batch* batch, const float* scores, const void* vision,
                             const void* text, const uint8_t* layer_mask,
                             const uint8_t* head_mask, const uint8_t* ffn_mask,
                             int32_t* kept_idx, float* resid, int32_t* cu_seqlens,
                             void* kv_cache, int32_t max_len, void* ws, size_t ws_bytes,
                             void* stream) {
  if (!kv_cache) return fail(SVL_E_NULL, "kv_cache is NULL");
  return prefill_impl(cfg, layers, batch, scores, vision, text, layer_mask, head_mask, ffn_mask,
                      kept_idx, resid, cu_seqlens, nullptr, ws, ws_bytes, stream, kv_cache, max_len);
}

svl_status svl_workspace_status(const void* ws, size_t ws_bytes, uint32_t* status, void* stream) {
  if (!ws || !status) return fail(SVL_E_NULL, "ws and status are required");
  if (!aligned16(ws)) return fail(SVL_E_ALIGN, "workspace not 16-byte aligned");
  if (ws_bytes < 256) return fail(SVL_E_WORKSPACE, "workspace of %zu bytes holds no status word", ws_bytes);
  const uint32_t* w = status_word(const_cast<void*>(ws), ws_bytes);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t v = 0;
  hipError_t e = hipMemcpyAsync(&v, w, sizeof(v), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "status read");
  *status = v;
  return SVL_OK;
}

size_t svl_kv_cache_bytes(const svl_config* cfg, int32_t batch, int32_t max_len) {
  if (check_config(cfg) != SVL_OK || batch <= 0 || max_len <= 0 || max_len > 32768) return 0;
  return (size_t)cfg->n_layers * batch * cfg->n_kv_heads * 2 * (size_t)max_len * cfg->head_dim * 2;
}

size_t svl_decode_workspace_bytes(const svl_config* cfg, int32_t batch, int32_t max_len) {
  if (check_config(cfg) != SVL_OK || batch <= 0 || max_len <= 0 || max_len > 32768) return 0;
  return (size_t)ws_layout(*cfg, batch, batch, max_len).total;
}

// Device scratch of svl_decode_step_noalloc: one copy per GPU, held until
// the process ends.  In host code `noalloc_scratch` names a host-side stand-in,
// not device memory: every host use goes through the device address that
// hipGetSymbolAddress returns on each GPU (scratch_address below).
static __device__ __align__(256) uint8_t noalloc_scratch[SVL_NOALLOC_SCRATCH_BYTES];

namespace svl {
namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the scratch array on the current GPU, looked up once per
// device (with that device current) and kept.
svl_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SVL_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SVL_E_HIP, "device index %d unsupported", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch));
    if (e != hipSuccess || !p)
      return fail(SVL_E_HIP, "scratch address on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SVL_OK;
}
}  // namespace
}  // namespace svl

// ws == nullptr: the allocation-free variant (the library's scratch array,
// the plan copied from pageable host memory).
static svl_status decode_impl(const svl_config* cfg, const svl_layer_weights* layers, int32_t batch,
                              float* x, const int32_t* cache_len, const uint8_t* layer_mask,
                              const uint8_t* head_mask, const uint8_t* ffn_mask, void* kv_cache,
                              int32_t max_len, void* ws, size_t ws_bytes, void* stream,
                              bool noalloc) {
  svl_status s = check_config(cfg);
  if (s != SVL_OK) return s;
  if (cfg->dtype != SVL_BF16) return fail(SVL_E_DTYPE, "decode runs on the 16-bit path only");
  if (batch <= 0) return fail(SVL_E_SHAPE, "batch must be positive");
  if (!x || !cache_len || !layer_mask || !head_mask || !kv_cache || (!noalloc && !ws))
    return fail(SVL_E_NULL, "NULL argument");
  if (!aligned16(x) || !aligned16(kv_cache) || (!noalloc && !aligned16(ws)))
    return fail(SVL_E_ALIGN, "device pointers must be 16-byte aligned");
  if (max_len <= 0 || max_len > 32768) return fail(SVL_E_SHAPE, "max_len outside [1, 32768]");
  for (int32_t b = 0; b < batch; ++b)
    if (cache_len[b] < 0 || cache_len[b] >= max_len)
      return fail(SVL_E_VALUE, "cache_len[%d] = %d outside [0, max_len)", b, cache_len[b]);
  const int32_t L = cfg->n_layers, A = cfg->n_heads, G = cfg->n_groups;
  if ((s = check_layers(*cfg, layers)) != SVL_OK) return s;
  if ((s = check_mask(layer_mask, (int64_t)batch * L, "layer_mask")) != SVL_OK) return s;
  if ((s = check_mask(head_mask, (int64_t)batch * L * A, "head_mask")) != SVL_OK) return s;
  if (ffn_mask && (s = check_mask(ffn_mask, (int64_t)batch * L * G, "ffn_mask")) != SVL_OK) return s;
  const WsLayout WL = ws_layout(*cfg, batch, batch, max_len);
  if (noalloc) {
    if (WL.total > (int64_t)SVL_NOALLOC_SCRATCH_BYTES)
      return fail(SVL_E_WORKSPACE,
                  "decode of %d samples with max_len %d needs %lld workspace bytes, the "
                  "allocation-free scratch holds %zu",
                  batch, max_len, (long long)WL.total, (size_t)SVL_NOALLOC_SCRATCH_BYTES);
    if ((s = scratch_address(&ws)) != SVL_OK) return s;
    ws_bytes = SVL_NOALLOC_SCRATCH_BYTES;
  }
  if ((int64_t)ws_bytes < WL.total)
    return fail(SVL_E_WORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)WL.total);
  std::vector<int32_t> seq(batch, 1);
  std::vector<LayerMasks> masks;
  std::vector<uint8_t> lon;
  layer_masks(*cfg, batch, layer_mask, head_mask, ffn_mask, masks, lon);
  std::string err;
  if (!build_plan(*cfg, batch, nullptr, seq.data(), L, masks.data(), &t_plan, &err, cache_len))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  Exec ex{*cfg, (hipStream_t)stream, static_cast<uint8_t*>(ws), WL, t_plan, x};
  ex.cache = static_cast<uint8_t*>(kv_cache);
  ex.max_len = max_len;
  ex.batch = batch;
  ex.decode = true;
  if ((s = stage(ex, true, noalloc)) != SVL_OK) return s;
  for (int32_t l = 0; l < L; ++l) {
    hipError_t e = ex.layer(t_plan.layers[l], layers[l], l);
    if (e != hipSuccess) return hip_fail(e, "layer launch");
  }
  hipError_t e = ex.norm(t_plan.final_norm, nullptr);
  if (e != hipSuccess) return hip_fail(e, "final residual launch");
  return SVL_OK;
}

svl_status svl_decode_step(const svl_config* cfg, const svl_layer_weights* layers, int32_t batch,
                           float* x, const int32_t* cache_len, const uint8_t* layer_mask,
                           const uint8_t* head_mask, const uint8_t* ffn_mask, void* kv_cache,
                           int32_t max_len, void* ws, size_t ws_bytes, void* stream) {
  return decode_impl(cfg, layers, batch, x, cache_len, layer_mask, head_mask, ffn_mask, kv_cache,
                     max_len, ws, ws_bytes, stream, false);
}

svl_status svl_decode_step_noalloc(const svl_config* cfg, const svl_layer_weights* layers,
                                   int32_t batch, float* x, const int32_t* cache_len,
                                   const uint8_t* layer_mask, const uint8_t* head_mask,
                                   const uint8_t* ffn_mask, void* kv_cache, int32_t max_len,
                                   void* stream) {
  return decode_impl(cfg, layers, batch, x, cache_len, layer_mask, head_mask, ffn_mask, kv_cache,
                     max_len, nullptr, 0, stream, true);
}

svl_status svl_count_positive(int32_t batch, int32_t n_vision, const float* logits,
                              int32_t* counts, void* ws, size_t ws_bytes, void* stream) {
  if (batch <= 0 || n_vision < 0) return fail(SVL_E_SHAPE, "batch must be positive, n_vision >= 0");
  if (!logits || !counts || !ws) return fail(SVL_E_NULL, "NULL argument");
  if (reinterpret_cast<uintptr_t>(logits) % 16 || reinterpret_cast<uintptr_t>(ws) % 16)
    return fail(SVL_E_VALUE, "device pointers must be 16-byte aligned");
  if (ws_bytes < (size_t)batch * 4) return fail(SVL_E_WORKSPACE, "workspace below 4 * batch bytes");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t* dev = static_cast<int32_t*>(ws);
  hipError_t e = launch_count_positive(logits, batch, n_vision, dev, st);
  if (e != hipSuccess) return hip_fail(e, "threshold count");
  e = hipMemcpyAsync(counts, dev, (size_t)batch * 4, hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return hip_fail(e, "threshold count copy");
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "threshold count sync");
  return SVL_OK;
}

svl_status svl_budget_project(const svl_config* cfg, int32_t batch, int32_t n_vision,
                              int32_t n_text, const int32_t* counts, float budget, int64_t vocab,
                              int32_t prefix, uint8_t* layer_mask, uint8_t* head_mask,
                              uint8_t* ffn_mask, const float* gate_logits, int32_t* keep) {
  svl_status s = check_config(cfg, false);
  if (s != SVL_OK) return s;
  if (batch <= 0 || n_vision < 0 || n_text < 0)
    return fail(SVL_E_SHAPE, "batch must be positive, token counts >= 0");
  if (!counts || !layer_mask || !head_mask || !keep) return fail(SVL_E_NULL, "NULL argument");
  if (!std::isfinite(budget) || !(budget > 0.f)) return fail(SVL_E_VALUE, "budget must be finite and > 0");
  if (vocab < 0) return fail(SVL_E_VALUE, "vocab must be >= 0");
  const int64_t L = cfg->n_layers, A = cfg->n_heads, G = cfg->n_groups;
  if (A % G) return fail(SVL_E_SHAPE, "n_heads %% n_groups != 0 (head groups)");
  if (prefix < 0 || prefix > L) return fail(SVL_E_VALUE, "prefix outside [0, n_layers]");
  if ((s = check_mask(layer_mask, batch * L, "layer_mask")) != SVL_OK) return s;
  if ((s = check_mask(head_mask, batch * L * A, "head_mask")) != SVL_OK) return s;
  if (ffn_mask && (s = check_mask(ffn_mask, batch * L * G, "ffn_mask")) != SVL_OK) return s;
  for (int32_t b = 0; b < batch; ++b)
    if (counts[b] < 0 || counts[b] > n_vision)
      return fail(SVL_E_VALUE, "counts[%d] = %d outside [0, %d]", b, counts[b], n_vision);
  if (gate_logits)
    for (int64_t i = 0; i < batch * L * G; ++i)
      if (!std::isfinite(gate_logits[i])) return fail(SVL_E_VALUE, "gate_logits[%lld] is not finite", (long long)i);
  for (int32_t b = 0; b < batch; ++b)
    keep[b] = project_budget_sample(*cfg, n_vision, n_text, counts[b], budget, vocab, prefix,
                                    layer_mask + b * L, head_mask + b * L * A,
                                    ffn_mask ? ffn_mask + b * L * G : nullptr,
                                    gate_logits ? gate_logits + b * L * G : nullptr, (int32_t)G);
  return SVL_OK;
}

// ------------------------------------------------------------ controlled prefill
// Workspace: the prefill's regions for the longest possible packing
// (B (N + T + 1) rows), then the controller's buffers.
struct CtrlLayout {
  int64_t counts, kappa, old_cu, kidx, pe, hid, eb, htil, glog, rcopy, total;
};

static CtrlLayout ctrl_layout(const svl_config& c, const svl_controller& k, int32_t B, int32_t N,
                              int32_t Rmax) {
  CtrlLayout L{};
  int64_t off = ws_layout(c, B, Rmax).total;
  auto take = [&](int64_t bytes) {
    const int64_t o = off;
    off = align256(off + std::max<int64_t>(bytes, 1));
    return o;
  };
  const int64_t E = k.pe_dim, H = k.hidden, D = c.d_model;
  const int64_t nl = (int64_t)(c.n_layers - k.prefix) * k.units;
  L.counts = take(4LL * B);
  L.kappa = take(8LL * B);
  L.old_cu = take(4LL * (B + 1));
  L.kidx = take(4LL * B * std::max(N, 1));
  L.pe = take(4LL * B * E);
  L.hid = take(4LL * B * H);
  L.eb = take(4LL * D);
  L.htil = take(4LL * B * D);
  L.glog = take(4LL * B * nl);
  L.rcopy = take(4LL * Rmax * D);
  take(256);   // the last bytes of the buffer hold the call's status word (svl_workspace_status)
  L.total = off;
  return L;
}

static svl_status check_controller(const svl_config& c, const svl_controller* k) {
  if (!k) return fail(SVL_E_NULL, "ctrl is NULL");
  if (k->prefix < 0 || k->prefix >= c.n_layers)
    return fail(SVL_E_VALUE, "ctrl->prefix %d outside [0, n_layers)", k->prefix);
  if (k->units != c.n_groups && k->units != 1)
    return fail(SVL_E_VALUE, "ctrl->units must be n_groups (layer-head) or 1 (layer)");
  if (k->units > 1 && c.n_heads % k->units)
    return fail(SVL_E_SHAPE, "n_heads %% n_groups != 0 (head groups)");
  if (k->pe_dim < 8 || k->pe_dim > 65536 || k->pe_dim % 8)
    return fail(SVL_E_SHAPE, "ctrl->pe_dim must be a multiple of 8 in [8, 65536]");
  if (k->hidden < 8 || k->hidden > 65536 || k->hidden % 8)
    return fail(SVL_E_SHAPE, "ctrl->hidden must be a multiple of 8 in [8, 65536]");
  if (c.d_model % 8) return fail(SVL_E_SHAPE, "the controller needs d_model %% 8 == 0");
  if (!std::isfinite(k->pe_scale)) return fail(SVL_E_VALUE, "ctrl->pe_scale must be finite");
  if (!std::isfinite(k->pe_base) || !(k->pe_base > 0.f))
    return fail(SVL_E_VALUE, "ctrl->pe_base must be finite and > 0");
  const void* w[10] = {k->llm_w1, k->llm_b1, k->llm_w2, k->llm_b2, k->kap_w1,
                       k->kap_b1, k->kap_w2, k->kap_b2, k->gate_w, k->gate_b};
  for (int i = 0; i < 10; ++i) {
    if (!w[i]) return fail(SVL_E_NULL, "NULL controller weight pointer");
    if (i % 2 == 0 && !aligned16(w[i]))
      return fail(SVL_E_ALIGN, "controller weight matrices must be 16-byte aligned");
  }
  return SVL_OK;
}

size_t svl_controlled_workspace_bytes(const svl_config* cfg, const svl_controller* ctrl,
                                      int32_t batch, int32_t n_vision, int32_t n_text) {
  if (check_config(cfg) != SVL_OK || check_controller(*cfg, ctrl) != SVL_OK) return 0;
  if (batch <= 0 || n_vision < 0 || n_text < 0) return 0;
  const int64_t rmax = (int64_t)batch * ((int64_t)n_vision + n_text + 1);
  if (rmax > INT32_MAX) return 0;
  return (size_t)ctrl_layout(*cfg, *ctrl, batch, n_vision, (int32_t)rmax).total;
}

svl_status svl_prefill_controlled(const svl_config* cfg, const svl_layer_weights* layers,
                                  const svl_controller* ctrl, int32_t batch, int32_t n_vision,
                                  int32_t n_text, float budget, int64_t vocab,
                                  const float* logits, const void* vision, const void* text,
                                  int32_t* kept_idx, float* resid, int32_t* cu_seqlens,
                                  int32_t* keep, uint8_t* layer_mask, uint8_t* head_mask,
                                  uint8_t* ffn_mask, float* gate_logits, svl_flops* flops,
                                  void* ws, size_t ws_bytes, void* stream) {
  svl_status s = check_config(cfg);
  if (s != SVL_OK) return s;
  const svl_config& c = *cfg;
  if ((s = check_layers(c, layers)) != SVL_OK) return s;
  if ((s = check_controller(c, ctrl)) != SVL_OK) return s;
  const svl_controller& k = *ctrl;
  if (batch <= 0 || n_vision < 0 || n_text < 0)
    return fail(SVL_E_SHAPE, "batch must be positive, token counts >= 0");
  if (!std::isfinite(budget) || !(budget > 0.f)) return fail(SVL_E_VALUE, "budget must be finite and > 0");
  if (vocab < 0) return fail(SVL_E_VALUE, "vocab must be >= 0");
  const int64_t rmax = (int64_t)batch * ((int64_t)n_vision + n_text + 1);
  if (rmax > INT32_MAX) return fail(SVL_E_SHAPE, "too many packed rows");
  if (!resid || !cu_seqlens || !keep || !layer_mask || !head_mask || !ffn_mask || !ws)
    return fail(SVL_E_NULL, "NULL argument");
  if (n_vision > 0 && (!logits || !vision || !kept_idx))
    return fail(SVL_E_NULL, "logits, vision and kept_idx are required when n_vision > 0");
  if (n_text > 0 && !text) return fail(SVL_E_NULL, "text is required when n_text > 0");
  for (const void* p : {(const void*)logits, vision, text, (const void*)kept_idx,
                        (const void*)resid, (const void*)ws})
    if (p && !aligned16(p)) return fail(SVL_E_ALIGN, "device pointers must be 16-byte aligned");
  const int32_t B = batch, N = n_vision, T = n_text, L = c.n_layers, A = c.n_heads;
  const int32_t G = c.n_groups, D = c.d_model, P = k.prefix, U = k.units;
  const int32_t E = k.pe_dim, H = k.hidden, nl = (L - P) * U, Rmax = (int32_t)rmax;
  const CtrlLayout CL = ctrl_layout(c, k, B, N, Rmax);
  if ((int64_t)ws_bytes < CL.total)
    return fail(SVL_E_WORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)CL.total);

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  int32_t* counts_dev = reinterpret_cast<int32_t*>(wsb + CL.counts);
  double* kappa_dev = reinterpret_cast<double*>(wsb + CL.kappa);
  int32_t* old_cu_dev = reinterpret_cast<int32_t*>(wsb + CL.old_cu);
  int32_t* kidx_dev = reinterpret_cast<int32_t*>(wsb + CL.kidx);
  float* pe_dev = reinterpret_cast<float*>(wsb + CL.pe);
  float* hid_dev = reinterpret_cast<float*>(wsb + CL.hid);
  float* eb_dev = reinterpret_cast<float*>(wsb + CL.eb);
  float* htil_dev = reinterpret_cast<float*>(wsb + CL.htil);
  float* glog_dev = reinterpret_cast<float*>(wsb + CL.glog);
  float* rcopy_dev = reinterpret_cast<float*>(wsb + CL.rcopy);
  const bool bf16 = c.dtype == SVL_BF16;
  auto linear = [&](const void* W, const void* bias, int32_t in, int32_t out, int32_t nvec,
                    int32_t act, const float* x, int64_t ldx, const float* add,
                    const int32_t* add_cu, float* y, int64_t ldy) {
    CtrlLinearArgs a{};
    a.W = W; a.bias = bias; a.in = in; a.out = out; a.nvec = nvec; a.act = act;
    a.x = x; a.ldx = ldx; a.add = add; a.add_cu = add_cu; a.ldadd = D; a.y = y; a.ldy = ldy;
    return timed(K_CTRL, st, [&] { return launch_ctrl_linear(a, bf16, st); });
  };
  hipError_t e;

  // 1. threshold counts and kappa
  e = timed(K_CTRL, st, [&] { return launch_ctrl_stats(logits, B, N, counts_dev, kappa_dev, st); });
  if (e != hipSuccess) return hip_fail(e, "controller statistics");
  std::vector<int32_t> counts(B);
  if ((e = hipMemcpyAsync(counts.data(), counts_dev, 4 * (size_t)B, hipMemcpyDeviceToHost, st)) !=
          hipSuccess ||
      (e = hipStreamSynchronize(st)) != hipSuccess)
    return hip_fail(e, "threshold counts");

  // 2. [kept vision ; text ; budget token] through the prefix layers at full capacity
  std::vector<int32_t> seq(B);
  int32_t R1 = 0;
  for (int32_t b = 0; b < B; ++b) { seq[b] = counts[b] + T + 1; R1 += seq[b]; }
  std::vector<uint8_t> all_on((size_t)B * A, 1);
  std::vector<LayerMasks> full(std::max(P, 1));
  for (auto& m : full) m = LayerMasks{all_on.data(), all_on.data(), A, nullptr, 0};
  std::string err;
  if (!build_plan(c, B, counts.data(), seq.data(), P, full.data(), &t_plan, &err))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  const WsLayout WL = ws_layout(c, B, Rmax);
  WsLayout WL1 = WL;
  WL1.partial_slice = (int64_t)R1 * D;
  Exec ex1{c, st, wsb, WL1, t_plan, resid};
  if ((s = stage(ex1, true)) != SVL_OK) return s;
  const int32_t* keep1_dev = ex1.at<int32_t>(t_plan.keep_off);
  const int32_t* cu1_dev = ex1.at<int32_t>(t_plan.cu_off);
  e = timed(K_SELECT, st, [&] { return launch_select(logits, B, N, keep1_dev, kidx_dev, st); });
  if (e == hipSuccess)
    e = timed(K_GATHER, st, [&] {
      return launch_gather(kidx_dev, keep1_dev, cu1_dev, B, N, T, D, R1, vision, text, c.dtype,
                           resid, st);
    });
  if (e == hipSuccess)
    e = timed(K_CTRL, st, [&] {
      return launch_pe(nullptr, (double)budget, 1, E, (double)k.pe_scale, (double)k.pe_base,
                       pe_dev, st);
    });
  if (e == hipSuccess)
    e = linear(k.llm_w1, k.llm_b1, E, H, 1, CTRL_ACT_GELU, pe_dev, E, nullptr, nullptr, hid_dev, H);
  if (e == hipSuccess)
    e = linear(k.llm_w2, k.llm_b2, H, D, 1, CTRL_ACT_NONE, hid_dev, H, nullptr, nullptr, eb_dev, D);
  if (e == hipSuccess)
    e = timed(K_CTRL, st, [&] { return launch_budget_rows(eb_dev, cu1_dev, B, D, resid, st); });
  for (int32_t l = 0; l < P && e == hipSuccess; ++l) e = ex1.layer(t_plan.layers[l], layers[l], l);
  if (e == hipSuccess) e = ex1.norm(t_plan.final_norm, nullptr);
  if (e != hipSuccess) return hip_fail(e, "prefix launch");

  // 3. gate logits: W_h (h_b^(P) + MLP_kappa(PE(kappa))) + c_h
  e = timed(K_CTRL, st, [&] {
    return launch_pe(kappa_dev, 0.0, B, E, (double)k.pe_scale, (double)k.pe_base, pe_dev, st);
  });
  if (e == hipSuccess)
    e = linear(k.kap_w1, k.kap_b1, E, H, B, CTRL_ACT_GELU, pe_dev, E, nullptr, nullptr, hid_dev, H);
  if (e == hipSuccess)
    e = linear(k.kap_w2, k.kap_b2, H, D, B, CTRL_ACT_NONE, hid_dev, H, resid, cu1_dev, htil_dev, D);
  if (e == hipSuccess)
    e = linear(k.gate_w, k.gate_b, D, nl, B, CTRL_ACT_NONE, htil_dev, D, nullptr, nullptr, glog_dev,
               nl);
  // the old packing's row offsets, kept for the compaction below
  if (e == hipSuccess)
    e = hipMemcpyAsync(old_cu_dev, cu1_dev, 4 * (size_t)(B + 1), hipMemcpyDeviceToDevice, st);
  std::vector<float> gl((size_t)B * nl);
  if (e == hipSuccess)
    e = hipMemcpyAsync(gl.data(), glog_dev, 4 * gl.size(), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "gate logits");
  for (size_t i = 0; i < gl.size(); ++i)
    if (!std::isfinite(gl[i])) return fail(SVL_E_VALUE, "gate logit %zu is not finite", i);

  // 4. masks (a unit is on iff its logit > 0), then the budget projection
  std::vector<float> conf((size_t)L * U, 0.f);
  std::vector<int32_t> keep2(counts);
  for (int32_t b = 0; b < B; ++b) {
    uint8_t* lm = layer_mask + (int64_t)b * L;
    uint8_t* hm = head_mask + (int64_t)b * L * A;
    uint8_t* fm = ffn_mask + (int64_t)b * L * G;
    const float* g = gl.data() + (size_t)b * nl;
    for (int32_t l = 0; l < L; ++l) {
      if (l < P) {
        lm[l] = 1;
        std::fill(hm + (int64_t)l * A, hm + (int64_t)(l + 1) * A, 1);
        std::fill(fm + (int64_t)l * G, fm + (int64_t)(l + 1) * G, 1);
        continue;
      }
      const float* gu = g + (size_t)(l - P) * U;
      if (U == 1) {
        const uint8_t on = gu[0] > 0.f ? 1 : 0;
        lm[l] = on;
        std::fill(hm + (int64_t)l * A, hm + (int64_t)(l + 1) * A, on);
        std::fill(fm + (int64_t)l * G, fm + (int64_t)(l + 1) * G, on);
      } else {
        uint8_t any = 0;
        const int32_t hg = A / G;
        for (int32_t j = 0; j < G; ++j) {
          const uint8_t on = gu[j] > 0.f ? 1 : 0;
          std::fill(hm + (int64_t)l * A + j * hg, hm + (int64_t)l * A + (j + 1) * hg, on);
          fm[(int64_t)l * G + j] = on;
          any |= on;
        }
        lm[l] = any;
      }
    }
    if (budget < 1.0f) {
      std::copy(g, g + nl, conf.begin() + (size_t)P * U);
      keep2[b] = project_budget_sample(c, N, T, counts[b], budget, vocab, P, lm, hm, fm,
                                       conf.data(), U);
    }
  }

  // 5. the discarded tokens leave at the prefix boundary; layers P..L-1
  bool compact = false;
  int32_t R2 = 0;
  for (int32_t b = 0; b < B; ++b) {
    compact = compact || keep2[b] < counts[b];
    seq[b] = keep2[b] + T + 1;
    R2 += seq[b];
  }
  if (compact &&
      (e = hipMemcpyAsync(rcopy_dev, resid, (size_t)R1 * D * 4, hipMemcpyDeviceToDevice, st)) !=
          hipSuccess)
    return hip_fail(e, "row copy");
  std::vector<LayerMasks> masks;
  std::vector<uint8_t> lon;
  layer_masks(c, B, layer_mask, head_mask, ffn_mask, masks, lon);
  if (!build_plan(c, B, keep2.data(), seq.data(), L - P, masks.data() + P, &t_plan, &err))
    return fail(SVL_E_VALUE, "%s", err.c_str());
  WsLayout WL2 = WL;
  WL2.partial_slice = (int64_t)R2 * D;
  Exec ex2{c, st, wsb, WL2, t_plan, resid};
  if ((s = stage(ex2, true)) != SVL_OK) return s;
  const int32_t* keep2_dev = ex2.at<int32_t>(t_plan.keep_off);
  const int32_t* cu2_dev = ex2.at<int32_t>(t_plan.cu_off);
  e = timed(K_SELECT, st, [&] { return launch_select(logits, B, N, keep2_dev, kept_idx, st); });
  if (e == hipSuccess && compact) {
    CompactArgs ca{rcopy_dev, resid, old_cu_dev, counts_dev, kidx_dev, cu2_dev, keep2_dev, kept_idx,
                   B, N, D};
    e = timed(K_CTRL, st, [&] { return launch_compact_rows(ca, R2, st); });
  }
  for (int32_t l = P; l < L && e == hipSuccess; ++l)
    e = ex2.layer(t_plan.layers[l - P], layers[l], l);
  if (e == hipSuccess) e = ex2.norm(t_plan.final_norm, nullptr);
  if (e != hipSuccess) return hip_fail(e, "layer launch");
  // the status word: cleared, then set if an output value is inf or NaN
  uint32_t* status = status_word(ws, ws_bytes);
  if ((e = launch_fill_i32(reinterpret_cast<int32_t*>(status), 0, 1, st)) != hipSuccess)
    return hip_fail(e, "status clear");
  if ((e = launch_nonfinite(resid, (int64_t)R2 * D, status, st)) != hipSuccess)
    return hip_fail(e, "status scan");

  cu_seqlens[0] = 0;
  for (int32_t b = 0; b < B; ++b) {
    cu_seqlens[b + 1] = cu_seqlens[b] + seq[b];
    keep[b] = keep2[b];
  }
  if (gate_logits) std::copy(gl.begin(), gl.end(), gate_logits);
  if (flops) {
    // prefix layers at the threshold lengths, the others at the final ones
    std::vector<uint8_t> lm1((size_t)B * L, 0), lm2(layer_mask, layer_mask + (size_t)B * L);
    std::vector<int32_t> seq1(B);
    for (int32_t b = 0; b < B; ++b) {
      seq1[b] = counts[b] + T + 1;
      for (int32_t l = 0; l < P; ++l) { lm1[(size_t)b * L + l] = 1; lm2[(size_t)b * L + l] = 0; }
    }
    svl_flops f1{}, f2{};
    if ((s = svl_count_flops(cfg, B, seq1.data(), lm1.data(), head_mask, ffn_mask, &f1)) != SVL_OK ||
        (s = svl_count_flops(cfg, B, seq.data(), lm2.data(), head_mask, ffn_mask, &f2)) != SVL_OK)
      return s;
    flops->q = f1.q + f2.q;
    flops->kv = f1.kv + f2.kv;
    flops->o = f1.o + f2.o;
    flops->attn = f1.attn + f2.attn;
    flops->ffn = f1.ffn + f2.ffn;
    flops->total = f1.total + f2.total;
  }
  return SVL_OK;
}

// ------------------------------------------------------------ training-time budget term
svl_status svl_budget_loss(const svl_config* cfg, const svl_budget_loss_params* p, int32_t batch,
                           int32_t n_vision, int32_t n_text, const float* logits,
                           const float* token_noise, const float* gate_logits,
                           const float* gate_noise, uint8_t* token_mask, uint8_t* unit_mask,
                           float* ratio, float* loss, float* grad_logits, float* grad_gate,
                           void* stream) {
  svl_status s = check_config(cfg, false);
  if (s != SVL_OK) return s;
  if (!p) return fail(SVL_E_NULL, "params is NULL");
  const svl_config& c = *cfg;
  if (batch <= 0 || n_vision < 0 || n_text < 0 || (int64_t)n_vision + n_text == 0)
    return fail(SVL_E_SHAPE, "batch must be positive, token counts >= 0 with n_vision + n_text > 0");
  if (p->prefix < 0 || p->prefix >= c.n_layers)
    return fail(SVL_E_VALUE, "prefix %d outside [0, n_layers)", p->prefix);
  if (p->units != c.n_groups && p->units != 1)
    return fail(SVL_E_VALUE, "units must be n_groups (layer-head) or 1 (layer)");
  if (p->vocab < 0) return fail(SVL_E_VALUE, "vocab must be >= 0");
  const float pos[3] = {p->budget, p->tau_tok, p->tau_comp};
  for (float v : pos)
    if (!std::isfinite(v) || !(v > 0.f))
      return fail(SVL_E_VALUE, "budget and temperatures must be finite and > 0");
  const float nonneg[4] = {p->margin, p->w_over, p->w_under, p->lambda_t};
  for (float v : nonneg)
    if (!std::isfinite(v) || v < 0.f)
      return fail(SVL_E_VALUE, "margin, loss weights and lambda must be finite and >= 0");
  if (!ratio || !loss || !gate_logits || !unit_mask || !grad_gate)
    return fail(SVL_E_NULL, "NULL argument");
  if (n_vision > 0 && (!logits || !token_mask || !grad_logits))
    return fail(SVL_E_NULL, "logits, token_mask and grad_logits are required when n_vision > 0");
  const double D = c.d_model, F = c.d_ffn, L = c.n_layers;
  const double Sf = (double)n_text + n_vision;
  BudgetLossArgs a{};
  a.z = logits; a.xi_tok = token_noise; a.gl = gate_logits; a.xi_gate = gate_noise;
  a.N = n_vision; a.T = n_text; a.L = c.n_layers; a.P = p->prefix; a.U = p->units;
  a.c1 = 8.0 * D * D + 6.0 * D * F;
  a.c2 = 4.0 * D;
  a.lm = 2.0 * D * (double)p->vocab;
  a.full = L * (a.c1 * Sf + a.c2 * Sf * Sf) + a.lm * Sf;
  a.budget = p->budget; a.margin = p->margin; a.w_over = p->w_over; a.w_under = p->w_under;
  a.lam = p->lambda_t; a.tau_comp = p->tau_comp;
  a.tok_mask = token_mask; a.unit_mask = unit_mask; a.ratio = ratio; a.loss = loss;
  a.grad_z = grad_logits; a.grad_gate = grad_gate;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(K_CTRL, st, [&] { return launch_budget_loss(a, batch, st); });
  if (e != hipSuccess) return hip_fail(e, "budget loss");
  return SVL_OK;
}

svl_status svl_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.on = on != 0;
  return SVL_OK;
}

svl_status svl_timing_read(int32_t kernel_class, double* total_ms, int64_t* launches) {
  if (kernel_class < 0 || kernel_class >= SVL_KCLASS_COUNT) return fail(SVL_E_VALUE, "bad kernel class");
  if (!total_ms || !launches) return fail(SVL_E_NULL, "NULL argument");
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double sum = 0.0;
  int64_t n = 0;
  std::vector<TimingRec> keep;
  for (auto& r : g_timing.recs) {
    if (r.cls != kernel_class) { keep.push_back(r); continue; }
    hipError_t e = hipEventSynchronize(r.b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(e, "timing read");
    sum += ms;
    ++n;
    g_timing.pool.push_back(r.a);
    g_timing.pool.push_back(r.b);
  }
  g_timing.recs.swap(keep);
  *total_ms = sum;
  *launches = n;
  return SVL_OK;
}

}  // extern "C"
