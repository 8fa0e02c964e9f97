// Host check of the launch planner (no GPU): for random batches, masks and
// shapes it builds the prefill plan and the decode plan and verifies, from
// the plan image alone,
//   * the image fits the bound the workspace reserves for it;
//   * QKV and gate/up tiles cover every (valid row, active head / K-V head /
//     FFN channel block) of every sample running the sub-block exactly once,
//     and nothing of an inactive one; a tile spanning several samples reads
//     its RoPE positions from the per-row table, which holds each row's
//     position inside its sample;
//   * output / down projection tiles give every (valid row, output block)
//     each active K chunk of its sample exactly once (summed over split-K
//     pieces), and no inactive chunk;
//   * decode of a batch: the shared row-vector segments give every (sample,
//     weight block) of an active head / K-V head / FFN slice exactly once,
//     and the output / down projections' use masks select exactly each
//     sample's active K chunks.
// Prints "plan_check ok" and exits 0, or reports the first violation.
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <string>
#include <tuple>
#include <vector>

#include "../paper_2607_20357_amd/csrc/plan.h"

using namespace svl;

static int g_fail = 0;
#define CHECK(c, ...)                                   \
  do {                                                  \
    if (!(c)) {                                         \
      std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      std::fprintf(stderr, __VA_ARGS__);                \
      std::fprintf(stderr, "\n");                       \
      if (++g_fail > 10) std::exit(1);                  \
    }                                                   \
  } while (0)

template <class T>
static const T* at(const Plan& p, int64_t off) {
  return reinterpret_cast<const T*>(p.image.data() + off);
}

struct Case {
  svl_config cfg;
  int32_t B;
  std::vector<int32_t> seq;
  std::vector<uint8_t> lon, hm, fm;   // [L][B], [L][B][A], [L][B][G]
  bool ffn_gated;
};

static std::vector<LayerMasks> masks_of(const Case& c) {
  std::vector<LayerMasks> m(c.cfg.n_layers);
  const int A = c.cfg.n_heads, G = c.cfg.n_groups, B = c.B;
  for (int l = 0; l < c.cfg.n_layers; ++l)
    m[l] = {c.lon.data() + (size_t)l * B, c.hm.data() + (size_t)l * B * A, A,
            c.ffn_gated ? c.fm.data() + (size_t)l * B * G : nullptr, G};
  return m;
}

// weight row of block gb of a paired / plain group (as the kernels compute it)
static int block_row(int kind, int wrow0, int gb, int d) {
  const int hb = d / 16;
  if (kind == 1) return wrow0 + (gb / hb) * d + (gb % hb) * 8;
  if (kind == 2) return wrow0 + gb * 8;
  return wrow0 + gb * 16;
}

static int g_waves4 = 0;   // launches planned with 4-wave tiles

static void check_prefill(const Case& c) {
  const svl_config& cfg = c.cfg;
  const int B = c.B, L = cfg.n_layers, A = cfg.n_heads, KV = cfg.n_kv_heads, d = cfg.head_dim;
  const int D = cfg.d_model, F = cfg.d_ffn, G = cfg.n_groups, rep = A / KV, slice = F / G;
  std::vector<int32_t> keep(c.seq);   // keep is only copied into the image
  auto masks = masks_of(c);
  Plan plan;
  std::string err;
  const bool ok = build_plan(cfg, B, keep.data(), c.seq.data(), L, masks.data(), &plan, &err);
  CHECK(ok, "build_plan: %s", err.c_str());
  if (!ok) return;
  int R = 0;
  std::vector<int> cu(B + 1, 0), pcu(B + 1, 0);
  for (int b = 0; b < B; ++b) {
    cu[b + 1] = cu[b] + c.seq[b];
    pcu[b + 1] = pcu[b] + (c.seq[b] + 15) / 16 * 16;
    R += c.seq[b];
  }
  CHECK((int64_t)plan.image.size() <= plan_bytes_bound(cfg, B, R, L), "image %zu > bound %lld",
        plan.image.size(), (long long)plan_bytes_bound(cfg, B, R, L));
  const int32_t* rowpos = at<int32_t>(plan, plan.rowpos_off);
  std::vector<int> sample_of(pcu[B], -1);
  for (int b = 0; b < B; ++b)
    for (int i = 0; i < c.seq[b]; ++i) {
      sample_of[pcu[b] + i] = b;
      CHECK(rowpos[pcu[b] + i] == i, "rowpos of sample %d row %d = %d", b, i, rowpos[pcu[b] + i]);
    }
  for (int l = 0; l < L; ++l) {
    const LayerPlan& LP = plan.layers[l];
    const LayerMasks& m = masks[l];
    const KChunk* chunks = at<KChunk>(plan, LP.chunks_off);
    auto runs_attn = [&](int b) {
      if (!m.layer_on[b] || c.seq[b] == 0) return false;
      for (int h = 0; h < A; ++h) if (m.head_mask[b * A + h]) return true;
      return false;
    };
    auto ffn_on = [&](int b, int j) { return !m.ffn_mask || m.ffn_mask[b * G + j]; };
    auto runs_ffn = [&](int b) {
      if (!m.layer_on[b] || c.seq[b] == 0) return false;
      for (int j = 0; j < G; ++j) if (ffn_on(b, j)) return true;
      return false;
    };
    // ---- QKV: count[(row, wsel, weight row of block)]
    std::map<std::tuple<int, int, int>, int> cnt;
    {
      const MmGroup* gr = at<MmGroup>(plan, LP.qkv.groups_off);
      const MmTile* tl = at<MmTile>(plan, LP.qkv.tiles_off);
      for (int t = 0; t < LP.qkv.ntiles; ++t) {
        const MmTile& x = tl[t];
        const MmGroup& g = gr[x.group];
        CHECK(x.arow % 16 == 0 && x.mcnt >= 1 && x.mcnt <= MFMA_BM, "qkv tile rows");
        CHECK(x.b0 >= 0 && x.b0 + x.nblk <= g.nblocks && x.nblk <= LP.qkv.nb, "qkv tile blocks");
        CHECK(LP.qkv.waves == 8 && LP.gu.waves == 8, "paired launches take 8-wave tiles");
        int s0 = -2;
        bool single = true;
        for (int r = 0; r < x.mcnt; ++r) {
          const int row = x.arow + r;
          CHECK(row < pcu[B], "qkv row past the padded rows");
          const int s = sample_of[row];
          if (s < 0) continue;
          if (s0 == -2) s0 = s;
          if (s != s0) single = false;
          if (x.pos0 >= 0) CHECK(x.pos0 + r == row - pcu[s], "qkv pos0 %d + %d != %d", x.pos0, r, row - pcu[s]);
          for (int j = 0; j < x.nblk; ++j) {
            const int wr = block_row(1, x.wrow0, x.b0 + j, d);
            ++cnt[{row, x.wsel, wr}];
          }
        }
        if (!single) CHECK(x.pos0 < 0, "a tile spanning samples must use the position table");
      }
      for (int b = 0; b < B; ++b)
        for (int i = 0; i < c.seq[b]; ++i) {
          const int row = pcu[b] + i;
          for (int sec = 0; sec < 3; ++sec) {
            const int n = sec == 0 ? A : KV;
            for (int h = 0; h < n; ++h) {
              bool on = runs_attn(b);
              if (on) {
                if (sec == 0) on = m.head_mask[b * A + h];
                else {
                  bool any = false;
                  for (int q = h * rep; q < (h + 1) * rep; ++q) any |= m.head_mask[b * A + q] != 0;
                  on = any;
                }
              }
              // blocks of head h: dims 8k .. 8k+7 with their rotary partners
              for (int k = 0; k < d / 16; ++k) {
                const int wr = h * d + k * 8;
                auto it = cnt.find({row, sec, wr});
                const int got = it == cnt.end() ? 0 : it->second;
                CHECK(got == (on ? 1 : 0), "qkv layer %d sample %d row %d sec %d head %d block %d: %d",
                      l, b, i, sec, h, k, got);
              }
            }
          }
        }
    }
    // ---- gate/up
    {
      std::map<std::pair<int, int>, int> cg;
      const MmGroup* gr = at<MmGroup>(plan, LP.gu.groups_off);
      const MmTile* tl = at<MmTile>(plan, LP.gu.tiles_off);
      for (int t = 0; t < LP.gu.ntiles; ++t) {
        const MmTile& x = tl[t];
        const MmGroup& g = gr[x.group];
        CHECK(x.b0 >= 0 && x.b0 + x.nblk <= g.nblocks && x.nblk <= LP.gu.nb, "gu tile blocks");
        for (int r = 0; r < x.mcnt; ++r) {
          const int row = x.arow + r;
          CHECK(row < pcu[B], "gu row past the padded rows");
          if (sample_of[row] < 0) continue;
          for (int j = 0; j < x.nblk; ++j) ++cg[{row, block_row(2, x.wrow0, x.b0 + j, d)}];
        }
      }
      for (int b = 0; b < B; ++b)
        for (int i = 0; i < c.seq[b]; ++i)
          for (int ch = 0; ch < F; ch += 8) {
            const bool on = runs_ffn(b) && ffn_on(b, ch / slice);
            auto it = cg.find({pcu[b] + i, ch});
            const int got = it == cg.end() ? 0 : it->second;
            CHECK(got == (on ? 1 : 0), "gu layer %d sample %d row %d channel %d: %d", l, b, i, ch, got);
          }
    }
    // ---- output / down projections: count[(residual row, output block, k0)]
    for (int which = 0; which < 2; ++which) {
      const GemmLaunch& GL = which == 0 ? LP.o : LP.down;
      const int K = which == 0 ? A * d : F;
      g_waves4 += GL.waves == 4;
      // 4-wave tiles only for unsplit 4-block launches with more tiles than CUs
      CHECK(GL.waves == 8 || (GL.waves == 4 && GL.nsplit == 1 && GL.nb == 4 &&
                              GL.ntiles > kTargetTiles),
            "plain launch waves %d (nsplit %d, nb %d, tiles %d)", GL.waves, GL.nsplit, GL.nb,
            GL.ntiles);
      std::map<std::tuple<int, int, int>, int> co;
      const MmGroup* gr = at<MmGroup>(plan, GL.groups_off);
      const MmTile* tl = at<MmTile>(plan, GL.tiles_off);
      for (int t = 0; t < GL.ntiles; ++t) {
        const MmTile& x = tl[t];
        const MmGroup& g = gr[x.group];
        CHECK(x.b0 >= 0 && x.b0 + x.nblk <= g.nblocks, "plain tile blocks");
        for (int r = 0; r < x.mcnt; ++r) {
          const int orow = x.orow + r;
          CHECK(orow < R, "plain output row past R");
          for (int j = 0; j < x.nblk; ++j)
            for (int cc = 0; cc < x.kcn; ++cc) {
              const int k0 = x.kdense >= 0 ? x.kdense + MFMA_BK * cc : chunks[x.chunk0 + cc].k0;
              CHECK(k0 >= 0 && k0 < K, "chunk outside K");
              ++co[{orow, x.b0 + j, k0}];
            }
        }
      }
      for (int b = 0; b < B; ++b) {
        const bool run = which == 0 ? runs_attn(b) : runs_ffn(b);
        for (int i = 0; i < c.seq[b]; ++i)
          for (int blk = 0; blk < D / 16; blk += 7)   // a sample of the blocks
            for (int k0 = 0; k0 < K; k0 += MFMA_BK) {
              bool on = run;
              if (on) on = which == 0 ? m.head_mask[b * A + k0 / d] != 0 : ffn_on(b, k0 / slice);
              auto it = co.find({cu[b] + i, blk, k0});
              const int got = it == co.end() ? 0 : it->second;
              CHECK(got == (on ? 1 : 0), "%s layer %d sample %d row %d block %d k0 %d: %d",
                    which == 0 ? "o" : "down", l, b, i, blk, k0, got);
            }
      }
    }
    // ---- attention tiles: each group's query tiles times its active query
    // heads, numbered consecutively; the group covers its sample's rows
    if (LP.attn.ntiles > 0) {
      const AttnGroup* ag = at<AttnGroup>(plan, LP.attn.groups_off);
      const int32_t* heads = at<int32_t>(plan, LP.attn.heads_off);
      const int bq = LP.attn.bq;
      CHECK(bq == ATTN_BQ || bq == ATTN_BQ_SHORT, "layer %d attention bq %d", l, bq);
      int tiles = 0;
      for (int gi = 0; gi < LP.attn.ngroups; ++gi) {
        const AttnGroup& g = ag[gi];
        CHECK(g.tile0 == tiles, "layer %d attention group %d tile0 %d != %d", l, gi, g.tile0, tiles);
        CHECK(g.sample >= 0 && g.sample < B && g.S == c.seq[g.sample] && g.row0 == pcu[g.sample],
              "layer %d attention group %d rows", l, gi);
        CHECK(g.nqt == (g.S + bq - 1) / bq, "layer %d attention group %d nqt %d", l, gi, g.nqt);
        CHECK(g.h_cnt >= 1 && g.kv_cnt >= 1, "layer %d attention group %d empty", l, gi);
        for (int i = 0; i < g.h_cnt; ++i)
          CHECK(m.head_mask[g.sample * A + heads[g.h_off + i]] != 0,
                "layer %d group %d lists inactive head %d", l, gi, heads[g.h_off + i]);
        tiles += g.nqt * g.h_cnt;
      }
      CHECK(tiles == LP.attn.ntiles, "layer %d attention tiles %d != %d", l, LP.attn.ntiles, tiles);
    }
  }
}

static void check_decode(const Case& c) {
  const svl_config& cfg = c.cfg;
  const int B = c.B, L = cfg.n_layers, A = cfg.n_heads, KV = cfg.n_kv_heads, d = cfg.head_dim;
  const int F = cfg.d_ffn, G = cfg.n_groups, rep = A / KV, slice = F / G;
  std::vector<int32_t> seq(B, 1), pos(B);
  for (int b = 0; b < B; ++b) pos[b] = c.seq[b];
  auto masks = masks_of(c);
  Plan plan;
  std::string err;
  const bool ok = build_plan(cfg, B, nullptr, seq.data(), L, masks.data(), &plan, &err, pos.data());
  CHECK(ok, "decode build_plan: %s", err.c_str());
  if (!ok) return;
  CHECK((int64_t)plan.image.size() <= plan_bytes_bound(cfg, B, B, L), "decode image %zu > bound %lld",
        plan.image.size(), (long long)plan_bytes_bound(cfg, B, B, L));
  if (B == 1) return;   // one sample: the per-group row-vector launches
  for (int l = 0; l < L; ++l) {
    const LayerPlan& LP = plan.layers[l];
    const LayerMasks& m = masks[l];
    const KChunk* chunks = at<KChunk>(plan, LP.chunks_off);
    auto runs = [&](int b, bool attn) {
      if (!m.layer_on[b]) return false;
      if (attn) { for (int h = 0; h < A; ++h) if (m.head_mask[b * A + h]) return true; return false; }
      for (int j = 0; j < G; ++j) if (!m.ffn_mask || m.ffn_mask[b * G + j]) return true;
      return false;
    };
    for (int cls = 0; cls < 4; ++cls) {
      const GemmLaunch& GL = cls == 0 ? LP.qkv : cls == 1 ? LP.o : cls == 2 ? LP.gu : LP.down;
      const bool attn = cls < 2;
      bool any = false;
      for (int b = 0; b < B; ++b) any |= runs(b, attn);
      CHECK(GL.nsegs > 0 || !any, "decode class %d has no segments", cls);
      const DecSeg* sg = at<DecSeg>(plan, GL.segs_off);
      const DecUse* us = at<DecUse>(plan, GL.uses_off);
      const int32_t* cm = at<int32_t>(plan, GL.cmasks_off);
      std::map<std::tuple<int, int, int, int>, int> cnt;   // (sample, wsel, weight row, k0)
      int blocks = 0;
      for (int s = 0; s < GL.nsegs; ++s) {
        const DecSeg& g = sg[s];
        CHECK(g.blk0 == blocks, "segments' blocks are consecutive");
        blocks += g.nblk;
        CHECK(g.nuse >= 1 && g.nuse <= DEC_MAX_USES && g.kc_cnt >= 1, "segment uses / chunks");
        CHECK(GL.max_uses >= g.nuse, "max_uses");
        for (int u = 0; u < g.nuse; ++u) {
          const int b = (us[g.use_off + u].arow) / 16;   // decode rows: one per sample, 16-row padded
          CHECK(us[g.use_off + u].arow == 16 * b, "use row");
          for (int gb = 0; gb < g.nblk; ++gb) {
            const int wr = block_row(cls == 0 ? 1 : cls == 2 ? 2 : 0, g.wrow0, gb, d);
            if (cls == 0 || cls == 2) {
              ++cnt[{b, g.wsel, wr, -1}];
            } else if (gb % 5 == 0) {   // a sample of the output blocks
              for (int cc = 0; cc < g.kc_cnt; ++cc) {
                const int mk = g.mask_off >= 0 ? cm[g.mask_off + cc] : -1;
                const int k0 = g.kdense >= 0 ? g.kdense + MFMA_BK * cc : chunks[g.kc_off + cc].k0;
                if ((mk >> u) & 1) ++cnt[{b, 0, wr, k0}];
              }
            }
          }
        }
      }
      CHECK(blocks == GL.nblocks, "segment blocks total");
      for (int b = 0; b < B; ++b) {
        const bool run = runs(b, attn);
        if (cls == 0) {
          for (int sec = 0; sec < 3; ++sec) {
            const int n = sec == 0 ? A : KV;
            for (int h = 0; h < n; ++h) {
              bool on = run;
              if (on) {
                if (sec == 0) on = m.head_mask[b * A + h];
                else {
                  bool a = false;
                  for (int q = h * rep; q < (h + 1) * rep; ++q) a |= m.head_mask[b * A + q] != 0;
                  on = a;
                }
              }
              for (int k = 0; k < d / 16; ++k) {
                auto it = cnt.find({b, sec, h * d + k * 8, -1});
                const int got = it == cnt.end() ? 0 : it->second;
                CHECK(got == (on ? 1 : 0), "decode qkv layer %d sample %d sec %d head %d: %d", l, b, sec, h, got);
              }
            }
          }
        } else if (cls == 2) {
          for (int ch = 0; ch < F; ch += 8) {
            const bool on = run && (!m.ffn_mask || m.ffn_mask[b * G + ch / slice]);
            auto it = cnt.find({b, 0, ch, -1});
            const int got = it == cnt.end() ? 0 : it->second;
            CHECK(got == (on ? 1 : 0), "decode gu layer %d sample %d channel %d: %d", l, b, ch, got);
          }
        } else {
          const int K = cls == 1 ? A * d : F;
          for (int wr = 0; wr < cfg.d_model; wr += 16 * 5)
            for (int k0 = 0; k0 < K; k0 += MFMA_BK) {
              bool on = run;
              if (on) on = cls == 1 ? m.head_mask[b * A + k0 / d] != 0
                                    : (!m.ffn_mask || m.ffn_mask[b * G + k0 / slice]);
              auto it = cnt.find({b, 0, wr, k0});
              const int got = it == cnt.end() ? 0 : it->second;
              CHECK(got == (on ? 1 : 0), "decode %s layer %d sample %d row %d k0 %d: %d",
                    cls == 1 ? "o" : "down", l, b, wr, k0, got);
            }
        }
      }
    }
  }
}

int main() {
  std::mt19937 rng(12345);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  int cases = 0;
  for (int it = 0; it < 60; ++it) {
    Case c{};
    const int d = U(0, 1) ? 64 : 128;
    const int KV = 1 << U(0, 2);
    const int rep = 1 << U(0, 2);
    const int A = KV * rep;
    const int G = A % 4 == 0 ? 4 : (A % 2 == 0 ? 2 : 1);
    const int D = 64 * U(2, 10);
    const int F = G * 64 * U(1, 4);
    c.cfg = svl_config{};
    c.cfg.n_layers = U(1, 3);
    c.cfg.d_model = D;
    c.cfg.n_heads = A;
    c.cfg.n_kv_heads = KV;
    c.cfg.head_dim = d;
    c.cfg.d_ffn = F;
    c.cfg.n_groups = G;
    c.cfg.rms_eps = 1e-6f;
    c.cfg.rope_theta = 10000.f;
    c.cfg.dtype = SVL_BF16;
    c.cfg.compute = SVL_COMPUTE_F16;
    c.B = it < 4 ? 1 : U(2, 19);
    c.seq.resize(c.B);
    for (int b = 0; b < c.B; ++b) c.seq[b] = U(0, 9) == 0 ? 0 : U(1, it % 3 == 0 ? 700 : 300);
    const int L = c.cfg.n_layers, B = c.B;
    c.lon.resize((size_t)L * B);
    c.hm.resize((size_t)L * B * A);
    c.fm.resize((size_t)L * B * G);
    c.ffn_gated = U(0, 3) != 0;
    const int pattern = U(0, 2);   // 0: random, 1: mostly shared masks, 2: whole groups
    for (int l = 0; l < L; ++l)
      for (int b = 0; b < B; ++b) {
        c.lon[(size_t)l * B + b] = U(0, 6) != 0;
        for (int h = 0; h < A; ++h) {
          uint8_t v;
          if (pattern == 0) v = U(0, 2) != 0;
          else if (pattern == 1) v = (h % 3 != 0) || U(0, 5) == 0;
          else v = ((h / (A / G)) + b + l) % 4 != 0;
          c.hm[((size_t)l * B + b) * A + h] = v;
        }
        for (int j = 0; j < G; ++j) {
          uint8_t v = pattern == 2 ? c.hm[((size_t)l * B + b) * A + j * (A / G)] : (uint8_t)(U(0, 3) != 0);
          c.fm[((size_t)l * B + b) * G + j] = v;
        }
      }
    check_prefill(c);
    check_decode(c);
    ++cases;
  }
  if (g_fail) {
    std::fprintf(stderr, "plan_check: %d failures\n", g_fail);
    return 1;
  }
  {
    // a batch whose output / down projections have more tiles than CUs
    // (16 samples x 3 M tiles x 8 N tiles)
    Case c{};
    c.cfg = svl_config{};
    c.cfg.n_layers = 1;
    c.cfg.d_model = 512;
    c.cfg.n_heads = 8;
    c.cfg.n_kv_heads = 8;
    c.cfg.head_dim = 64;
    c.cfg.d_ffn = 256;
    c.cfg.n_groups = 4;
    c.cfg.rms_eps = 1e-6f;
    c.cfg.rope_theta = 10000.f;
    c.cfg.dtype = SVL_BF16;
    c.cfg.compute = SVL_COMPUTE_F16;
    c.B = 16;
    c.seq.assign(c.B, 520);
    c.lon.assign(c.B, 1);
    c.hm.assign((size_t)c.B * 8, 1);
    c.fm.assign((size_t)c.B * 4, 1);
    c.ffn_gated = true;
    check_prefill(c);
    ++cases;
  }
  if (g_waves4 == 0) {
    std::fprintf(stderr, "plan_check: no case planned 4-wave tiles\n");
    return 1;
  }
  std::printf("plan_check ok (%d cases, %d launches with 4-wave tiles)\n", cases, g_waves4);
  return 0;
}
