// Host planner.  For each layer it lists, per executed sample:
//   * the rows whose residual is finished and normed before each sub-block
//     (adding pending split-K partial slices, writing the normed rows);
//   * the active output-column ranges of the QKV and gate/up GEMMs (only
//     active heads' and active FFN slices' weight rows are ever read);
//   * the active K chunks of the output and down projections (only active
//     heads' / slices' weight columns are ever read);
//   * the active heads of the attention launch.
// On the 16-bit MFMA path it also cuts every GEMM launch into a tile table:
// the QKV and gate/up launches spread their column blocks evenly over about
// one tile per CU; the output and down projections use 4-block tiles and,
// for skinny samples, split K so the launch still covers the CUs.
#include "plan.h"

#include <algorithm>
#include <cstdlib>
#include <cstring>

namespace svl {
namespace {

int64_t align16(int64_t x) { return (x + 15) & ~int64_t(15); }

struct ImageWriter {
  std::vector<uint8_t>* img;
  template <class T>
  int64_t append(const std::vector<T>& v) {
    int64_t off = align16((int64_t)img->size());
    img->resize(off + (int64_t)(v.size() * sizeof(T)));
    if (!v.empty()) std::memcpy(img->data() + off, v.data(), v.size() * sizeof(T));
    return off;
  }
  // room for n records of T at the end of the image (filled by the caller
  // through at<T>() before the next append)
  template <class T>
  int64_t reserve(int64_t n) {
    int64_t off = align16((int64_t)img->size());
    img->resize(off + n * (int64_t)sizeof(T));
    return off;
  }
  template <class T>
  T* at(int64_t off) { return reinterpret_cast<T*>(img->data() + off); }
};

struct Range {
  int32_t a, b;
};

// Maximal runs of set entries of m[0..n) scaled by `unit`, shifted by `base`.
std::vector<Range> runs(const uint8_t* m, int32_t n, int32_t unit, int32_t base) {
  std::vector<Range> r;
  int32_t i = 0;
  while (i < n) {
    if (!m[i]) { ++i; continue; }
    int32_t j = i;
    while (j < n && m[j]) ++j;
    r.push_back({base + i * unit, base + j * unit});
    i = j;
  }
  return r;
}

int32_t cdiv(int32_t a, int32_t b) { return (a + b - 1) / b; }

struct GemmBuild {
  std::vector<GemmGroup> groups;
  int32_t max_rows = 0, min_chunks = 1 << 30;
  void add(int32_t arow0, int32_t orow0, int32_t nrows, int32_t n0, int32_t n1, int32_t kc_off,
           int32_t kc_cnt) {
    if (nrows <= 0 || n1 <= n0 || kc_cnt <= 0) return;
    GemmGroup g{};
    g.arow0 = arow0; g.orow0 = orow0; g.nrows = nrows; g.n0 = n0; g.n1 = n1;
    g.kc_off = kc_off; g.kc_cnt = kc_cnt; g.nsplit = 1;
    groups.push_back(g);
    max_rows = std::max(max_rows, nrows);
    min_chunks = std::min(min_chunks, kc_cnt);
  }
  int32_t out_tiles(int32_t BM, int32_t BNO) const {
    int32_t t = 0;
    for (const auto& g : groups) t += cdiv(g.nrows, BM) * cdiv(g.n1 - g.n0, BNO);
    return t;
  }
  // Numbers the tiles (split fastest, then M tile, then N tile) for tiles of
  // BM rows x BNO output columns; bn is the tile width in weight rows.
  GemmLaunch finish(ImageWriter& w, int32_t BM, int32_t BNO, int32_t bn, int32_t nsplit) {
    GemmLaunch L;
    int32_t tile = 0;
    for (auto& g : groups) {
      g.nsplit = nsplit;
      g.tile0 = tile;
      tile += nsplit * cdiv(g.nrows, BM) * cdiv(g.n1 - g.n0, BNO);
    }
    L.groups_off = w.append(groups);
    L.ngroups = (int32_t)groups.size();
    L.ntiles = tile;
    L.nb = bn;
    L.nsplit = nsplit;
    return L;
  }
};

// 16-bit MFMA GEMM launch: groups, then the tile table.
struct MmBuild {
  std::vector<MmGroup> groups;
  int32_t max_rows = 0, min_chunks = 1 << 30;
  void add(int32_t arow0, int32_t orow0, int32_t nrows, int32_t wsel, int32_t wrow0,
           int32_t ocol0, int32_t nblocks, int32_t kc_off, int32_t kc_cnt, int32_t rope,
           const std::vector<KChunk>& chunks, int32_t pos_base = 0) {
    if (nrows <= 0 || nblocks <= 0 || kc_cnt <= 0) return;
    MmGroup g{};
    g.pos_base = pos_base;
    g.arow0 = arow0; g.orow0 = orow0; g.nrows = nrows; g.wsel = wsel; g.wrow0 = wrow0;
    g.ocol0 = ocol0; g.kc_off = kc_off; g.kc_cnt = kc_cnt; g.rope = rope; g.nblocks = nblocks;
    // contiguous full chunks: the kernel computes the offsets
    g.kdense = chunks[kc_off].k0;
    for (int32_t c = 0; c < kc_cnt; ++c)
      if (chunks[kc_off + c].k0 != g.kdense + MFMA_BK * c || chunks[kc_off + c].len != MFMA_BK) {
        g.kdense = -1;
        break;
      }
    groups.push_back(g);
    max_rows = std::max(max_rows, nrows);
    min_chunks = std::min(min_chunks, kc_cnt);
    max_chunks = std::max(max_chunks, kc_cnt);
  }
  int32_t max_chunks = 0;
  // (group, M tile) pairs' total block count
  int64_t total_blocks() const {
    int64_t tb = 0;
    for (const auto& g : groups) tb += (int64_t)cdiv(g.nrows, MFMA_BM) * g.nblocks;
    return tb;
  }
  // Tiles of `bpt` blocks at most, the blocks of a (group, M tile) split
  // evenly; tiles that share weight blocks (M tiles) and split-K pieces are
  // consecutive, so they land on one XCD.
  GemmLaunch finish(ImageWriter& w, int32_t bpt, int32_t nb, int32_t nsplit) {
    GemmLaunch L;
    for (auto& g : groups) {   // block numbering of the row-vector launches
      g.pad0 = L.nblocks;
      L.nblocks += g.nblocks;
    }
    L.groups_off = w.append(groups);
    int64_t count = 0;
    for (const auto& g : groups)
      count += (int64_t)cdiv(g.nblocks, bpt) * cdiv(g.nrows, MFMA_BM) * nsplit;
    L.tiles_off = w.reserve<MmTile>(count);
    MmTile* out = w.at<MmTile>(L.tiles_off);
    int64_t n = 0;
    int32_t kc[MFMA_MAX_SPLIT + 1];
    for (int32_t gi = 0; gi < (int32_t)groups.size(); ++gi) {
      const MmGroup& g = groups[gi];
      const int32_t nt = cdiv(g.nblocks, bpt), nm = cdiv(g.nrows, MFMA_BM);
      for (int32_t p = 0; p <= nsplit; ++p) kc[p] = (int32_t)((int64_t)g.kc_cnt * p / nsplit);
      MmTile t{};   // the fields shared by the group's tiles
      t.wsel = g.wsel; t.wrow0 = g.wrow0; t.ocol0 = g.ocol0; t.rope = g.rope; t.group = gi;
      int32_t b0 = 0;
      for (int32_t q = 0; q < nt; ++q) {
        const int32_t b1 = (int32_t)((int64_t)(q + 1) * g.nblocks / nt);
        t.b0 = b0; t.nblk = b1 - b0;
        for (int32_t mt = 0; mt < nm; ++mt) {
          const int32_t m0 = mt * MFMA_BM;
          t.arow = g.arow0 + m0;
          t.orow = g.orow0 + m0;
          t.mcnt = std::min(MFMA_BM, g.nrows - m0);
          t.pos0 = g.pos_base >= 0 ? g.pos_base + m0 : -1;
          for (int32_t p = 0; p < nsplit; ++p) {
            t.chunk0 = g.kc_off + kc[p];
            t.kcn = kc[p + 1] - kc[p];
            t.kdense = g.kdense >= 0 ? g.kdense + MFMA_BK * kc[p] : -1;
            t.slice = p;
            out[n++] = t;
          }
        }
        b0 = b1;
      }
    }
    L.ngroups = (int32_t)groups.size();
    L.ntiles = (int32_t)count;
    L.nb = nb;
    L.nsplit = nsplit;
    return L;
  }
  int64_t tiles_for(int32_t bpt) const {
    int64_t n = 0;
    for (const auto& g : groups) n += (int64_t)cdiv(g.nrows, MFMA_BM) * cdiv(g.nblocks, bpt);
    return n;
  }
  // QKV and gate/up: blocks per tile (and split-K pieces) by a cost model of
  // the launch time.  A CU's vector memory path keeps a bounded number of
  // cache lines in flight, so a tile costs (lines it loads) x (their
  // latency): per K chunk, one 128-byte line per activation row (L2 hits,
  // ~280 cycles) and one per weight row (HBM, ~1400 cycles).  The launch
  // costs (rounds of one tile per CU) x (the widest tile), plus, when split,
  // the finish kernel that reads the float32 slices back (~3 us fixed).
  // Splitting cuts each tile's activation lines; wider tiles cut the number
  // of tiles that all stream the same activations.
  //
  // Measured on the headline shapes, splitting does not pay: wider tiles
  // stop hiding their MFMA work behind the loads and the finish costs a
  // launch, so splitting is off unless forced (`force_split` > 1, from the
  // SVL_PAIRED_SPLIT environment variable: tuning and tests).
  GemmLaunch finish_paired(ImageWriter& w, int32_t pld, int64_t cap_floats, int32_t prows,
                           int32_t items_per_block, int32_t force_split) {
    const double rows = (double)std::min<int64_t>(MFMA_BM, max_rows);
    int32_t best_b = 1, best_s = 1;
    double best_t = -1.0;
    // a forced split applies to skinny launches and only while it needs no
    // more tiles than one per CU (the plan image is sized for that)
    const int32_t s_lo = (force_split > 1 && max_rows <= kSkinnyRows) ? force_split : 1;
    const int32_t s_hi = s_lo;
    for (int32_t s = s_lo; s <= s_hi; ++s) {
      if (s > 1 && (min_chunks < 4 * s || (int64_t)s * prows * pld > cap_floats)) break;
      for (int32_t bpt = 1; bpt <= MFMA_MAX_NB; ++bpt) {
        const int64_t rounds = (tiles_for(bpt) * s + kTargetTiles - 1) / kTargetTiles;
        const double kcn = (double)max_chunks / s;
        const double tile_us = kcn * (rows * 280.0 + 16.0 * bpt * 1400.0) / 90.0 / 2400.0;
        const double t = (double)rounds * tile_us;
        if (best_t < 0 || t < best_t - 1e-9) { best_b = bpt; best_s = s; best_t = t; }
      }
    }
    if (best_s > 1 && tiles_for(best_b) * best_s > kTargetTiles) {
      best_s = 1;
      best_t = -1.0;
      for (int32_t bpt = 1; bpt <= MFMA_MAX_NB; ++bpt) {
        const int64_t rounds = (tiles_for(bpt) + kTargetTiles - 1) / kTargetTiles;
        const double t = (double)rounds * max_chunks * (rows * 280.0 + 16.0 * bpt * 1400.0) / 216000.0;
        if (best_t < 0 || t < best_t - 1e-9) { best_b = bpt; best_t = t; }
      }
    }
    if (best_s > 1) {
      int32_t item = 0;
      for (auto& g : groups) {
        g.fitem0 = item;
        item += g.nrows * g.nblocks * items_per_block;
      }
      GemmLaunch L = finish(w, best_b, kernel_nb(best_b), best_s);
      L.nitems = item;
      return L;
    }
    // the smallest block count with the same number of rounds
    const int64_t rounds = (tiles_for(best_b) + kTargetTiles - 1) / kTargetTiles;
    while (best_b > 1 && (tiles_for(best_b - 1) + kTargetTiles - 1) / kTargetTiles == rounds)
      --best_b;
    return finish(w, best_b, kernel_nb(best_b), 1);
  }
  // Output and down projections: 4-block tiles; a skinny launch splits K
  // into float32 partial slices (at least 2 chunks per piece, the slices
  // within the partial buffer).
  GemmLaunch finish_plain(ImageWriter& w, int32_t R, int32_t D, int64_t cap_floats,
                          bool rowvec = false) {
    int32_t s = 1;
    if (!rowvec && !groups.empty() && max_rows <= kSkinnyRows) {
      int64_t base = 0;
      for (const auto& g : groups) base += (int64_t)cdiv(g.nrows, MFMA_BM) * cdiv(g.nblocks, 4);
      s = (int32_t)std::max<int64_t>(1, kTargetTiles / std::max<int64_t>(1, base));
      s = std::min(s, MFMA_MAX_SPLIT);
      s = std::min(s, std::max(1, min_chunks / 2));
      s = std::min<int64_t>(s, std::max<int64_t>(1, cap_floats / ((int64_t)std::max(1, R) * D)));
    }
    GemmLaunch L = finish(w, 4, 4, s);
    // more tiles than CUs: 4-wave tiles, two per CU (measured 20% faster per
    // launch on the ragged batch of 8; slower for one tile per CU)
    if (!rowvec && s == 1 && L.ntiles > kTargetTiles) L.waves = 4;
    return L;
  }
  // kernel instantiations: 2, 3, 4, 5, 6, 8 blocks (a tile's unused blocks
  // still cost their MFMAs, so the kernel is the smallest that fits)
  static int32_t kernel_nb(int32_t bpt) { return bpt <= 2 ? 2 : (bpt <= 6 ? bpt : 8); }
};

// K chunks covering [a, b) in pieces of at most `bk` columns.
void push_chunks(std::vector<KChunk>& ch, int32_t a, int32_t b, int32_t bk) {
  for (int32_t k = a; k < b; k += bk) ch.push_back({k, std::min(bk, b - k)});
}

// Shared row-vector launch of one layer's GEMM (decode of a batch):
// segments of weight blocks with the samples that use them.
struct DecBuild {
  std::vector<DecSeg> segs;
  std::vector<DecUse> uses;
  std::vector<int32_t> masks;
  int32_t nblocks = 0, max_uses = 0;
  // One segment per group of at most DEC_MAX_USES samples; `masks_of(c)`
  // gives chunk c's use mask for the group's samples (empty: every use).
  void add(int32_t nblk, int32_t wsel, int32_t wrow0, int32_t ocol0, int32_t rope,
           const std::vector<int32_t>& samples, const std::vector<int32_t>& arow,
           const std::vector<int32_t>& orow, const int32_t* pos, int32_t kc_off, int32_t kc_cnt,
           int32_t kdense, const std::vector<int32_t>* per_sample_chunk_on = nullptr,
           int32_t nchunks_all = 0, std::vector<KChunk>* chunks = nullptr) {
    for (size_t s0 = 0; s0 < samples.size(); s0 += DEC_MAX_USES) {
      const size_t s1 = std::min(samples.size(), s0 + DEC_MAX_USES);
      DecSeg g{};
      g.blk0 = nblocks; g.nblk = nblk; g.wsel = wsel; g.wrow0 = wrow0; g.ocol0 = ocol0;
      g.rope = rope; g.nuse = (int32_t)(s1 - s0); g.use_off = (int32_t)uses.size();
      g.kc_off = kc_off; g.kc_cnt = kc_cnt; g.kdense = kdense; g.mask_off = -1;
      for (size_t i = s0; i < s1; ++i) {
        const int32_t b = samples[i];
        uses.push_back({arow[b], orow[b], pos ? pos[b] : 0, 0});
      }
      if (per_sample_chunk_on) {
        // the union of the group's active chunks, each with its use mask
        g.kc_off = (int32_t)chunks->size();
        g.mask_off = (int32_t)masks.size();
        g.kdense = -1;
        for (int32_t c = 0; c < nchunks_all; ++c) {
          int32_t mk = 0;
          for (size_t i = s0; i < s1; ++i)
            if ((*per_sample_chunk_on)[(size_t)samples[i] * nchunks_all + c]) mk |= 1 << (i - s0);
          if (!mk) continue;
          chunks->push_back({c * MFMA_BK, MFMA_BK});
          masks.push_back(mk);
        }
        g.kc_cnt = (int32_t)chunks->size() - g.kc_off;
        if (g.kc_cnt == 0) continue;
      }
      segs.push_back(g);
      nblocks += nblk;
      max_uses = std::max(max_uses, g.nuse);
    }
  }
  void finish(ImageWriter& w, GemmLaunch& L) {
    if (segs.empty()) return;
    L.segs_off = w.append(segs);
    L.uses_off = w.append(uses);
    L.cmasks_off = w.append(masks);
    L.nsegs = (int32_t)segs.size();
    L.nblocks = nblocks;
    L.max_uses = max_uses;
  }
};

}  // namespace

int64_t plan_bytes_bound(const svl_config& c, int32_t B, int32_t R, int32_t nlayers) {
  const int64_t A = c.n_heads, KV = c.n_kv_heads, G = c.n_groups, d = c.head_dim;
  const int64_t F = c.d_ffn, D = c.d_model;
  const int64_t bk = 64;
  // M tiles over all samples: sum of ceil(S_b / BM) <= B + R / BM
  const int64_t mts = B + (int64_t)R / MFMA_BM + 1;
  auto tile_bound = [&](int64_t groups, int64_t blocks) {
    // (group, M tile) pairs + max(one launch's CU target, blocks / MFMA_MAX_NB);
    // a split launch keeps its tile count at the CU target
    const int64_t pairs = groups * mts;
    const int64_t tb = mts * blocks;
    return (pairs + std::max<int64_t>(kTargetTiles, tb / MFMA_MAX_NB + 1) +
            std::max<int64_t>(kTargetTiles, mts * ((blocks + 3) / 4))) *
               (int64_t)sizeof(MmTile) + 32;
  };
  int64_t per_layer = 0;
  per_layer += 2 * (B * (int64_t)sizeof(NormSeg) + 16);
  // QKV: at most one range per head (q) and per kv head (k and v)
  const int64_t gsz = std::max<int64_t>(sizeof(GemmGroup), sizeof(MmGroup));
  per_layer += B * (A + 2 * KV) * gsz + 16;
  per_layer += B * gsz + 16;                 // o
  per_layer += B * G * gsz + 16;             // gate/up
  per_layer += B * gsz + 16;                 // down
  per_layer += tile_bound(B * (A + 2 * KV), (A + 2 * KV) * d / 16);
  per_layer += tile_bound(B, D / 16);
  per_layer += tile_bound(B * G, F / 8);
  per_layer += tile_bound(B, D / 16);
  per_layer += B * (int64_t)sizeof(AttnGroup) + 16;
  per_layer += B * A * 4 + 16;
  per_layer += B * KV * 4 + 16;              // active K/V heads (cache append)
  // chunks: dense D, per sample active head columns and FFN slices
  int64_t chunks = (D + bk - 1) / bk + B * A * ((d + bk - 1) / bk) +
                   B * G * ((F / G + bk - 1) / bk);
  per_layer += chunks * (int64_t)sizeof(KChunk) + 16;
  // shared row-vector segments (decode of a batch): at most one segment per
  // (head, K/V head, FFN slice or projection) and group of DEC_MAX_USES
  // samples, one use per sample in each, and the output / down projections'
  // union chunk lists with their use masks
  const int64_t ngrp = (B + DEC_MAX_USES - 1) / DEC_MAX_USES;
  const int64_t nseg = (A + 2 * KV + G + 2) * ngrp;
  const int64_t nuch = 2 * ngrp * ((A * d + F) / bk + 2);
  per_layer += nseg * (int64_t)sizeof(DecSeg) + (A + 2 * KV + G + 2) * B * (int64_t)sizeof(DecUse) +
               nuch * (int64_t)(sizeof(KChunk) + 4) + 64;
  // per activation row: the position table
  const int64_t row_tables = 4 * ((int64_t)R + 16 * B + 1) + 16;
  return 64 + row_tables + (int64_t)B * 4 + (int64_t)(B + 1) * 4 + 32 + B * (int64_t)sizeof(NormSeg) + 16 +
         per_layer * nlayers;
}

bool build_plan(const svl_config& cfg, int32_t B, const int32_t* keep, const int32_t* seqlens,
                int32_t nlayers, const LayerMasks* masks, Plan* plan, std::string* err,
                const int32_t* pos_base) {
  const bool mfma = cfg.dtype == SVL_BF16;
  // decode (cached positions given): one row per sample, so the 16-bit GEMMs
  // run as row-vector launches over the groups' blocks and the output / down
  // projections add straight into the residual (no split-K)
  const bool rowvec = pos_base != nullptr;
  const int32_t A = cfg.n_heads, KV = cfg.n_kv_heads, G = cfg.n_groups, d = cfg.head_dim;
  const int32_t D = cfg.d_model, F = cfg.d_ffn, rep = A / KV, slice = F / G;
  const int32_t BM = mfma ? MFMA_BM : F32_BM;
  const int32_t bk = 64;

  plan->image.clear();
  plan->layers.assign(nlayers, LayerPlan{});
  plan->final_norm = NormLaunch{};
  plan->max_seq = 0;
  plan->max_pos = 0;
  ImageWriter w{&plan->image};

  std::vector<int32_t> cu(B + 1, 0), pcu(B + 1, 0);
  for (int32_t b = 0; b < B; ++b) {
    if (seqlens[b] < 0) { *err = "negative sequence length"; return false; }
    cu[b + 1] = cu[b] + seqlens[b];
    pcu[b + 1] = pcu[b] + (mfma ? (seqlens[b] + 15) / 16 * 16 : seqlens[b]);
    plan->max_seq = std::max(plan->max_seq, seqlens[b]);
    const int32_t pb = pos_base ? pos_base[b] : 0;
    if (pb < 0) { *err = "negative cached length"; return false; }
    plan->max_pos = std::max(plan->max_pos, pb + seqlens[b]);
  }
  const int32_t R = cu[B];
  plan->padded_rows = pcu[B];
  if (mfma && (int64_t)plan->max_seq * (A + 2 * KV) * d * 2 >= (int64_t(1) << 31)) {
    *err = "a sample's Q/K/V rows span 2 GiB or more (attention addresses them with 32-bit offsets)";
    return false;
  }
  // split-K partial slices the workspace holds (decode: none, it never splits)
  const int64_t cap = rowvec ? 0 : partial_floats_bound(cfg, B, R);
  int32_t force_split = 1;
  if (const char* e = std::getenv("SVL_PAIRED_SPLIT")) force_split = std::max(1, std::min(4, std::atoi(e)));
  // 8-row-group norm kernel: 16-bit output, d_model % 256 == 0 and <= 8192
  // (a row in one wave's registers); SVL_NORM8_MIN_ROWS overrides the row
  // threshold (tuning and tests)
  int32_t rows8_min = kNormRows8;
  if (const char* e = std::getenv("SVL_NORM8_MIN_ROWS")) rows8_min = std::max(0, std::atoi(e));
  const bool rows8_ok = mfma && D % 256 == 0 && D <= 8192;
  const int32_t qkv_width = (A + 2 * KV) * d;
  std::vector<int32_t> kp(B, 0);
  if (keep) for (int32_t b = 0; b < B; ++b) kp[b] = keep[b];
  plan->keep_off = w.append(kp);
  plan->cu_off = w.append(cu);
  {
    std::vector<int32_t> rp(std::max<int32_t>(1, pcu[B]), 0);
    for (int32_t b = 0; b < B; ++b)
      for (int32_t i = 0; i < seqlens[b]; ++i) rp[(size_t)pcu[b] + i] = (pos_base ? pos_base[b] : 0) + i;
    plan->rowpos_off = w.append(rp);
  }
  // 16-bit prefill of a batch: QKV and gate/up groups span runs of
  // consecutive samples that share a head, K/V head or FFN slice, so a shared
  // weight block is streamed once per 256 rows of the run instead of once per
  // sample; rows between samples are padding rows whose results land in
  // padding rows of the GEMM's own output buffer.  (Output / down projection
  // groups spanning samples with identical active sets measured 0.4-6 us
  // slower per launch on the batch workloads, so they stay per sample.)
  const bool span = mfma && !pos_base && B > 1 && force_split <= 1;

  // samples whose residual rows wait for split-K partial slices
  std::vector<uint8_t> pending(B, 0);
  int32_t pending_split = 0;

  // A residual / norm launch over the samples that are pending or run the
  // next sub-block (run[b] != 0).
  // A sub-block that no sample runs launches nothing: split-K partials still
  // pending (from the last output / down projection) stay in their slices,
  // untouched until the next sub-block a sample runs, whose norm adds them
  // (`final`: the closing add-only launch after the last layer).
  auto norm_launch = [&](const std::vector<uint8_t>& run, bool final = false) {
    NormLaunch L;
    bool any = final;
    for (int32_t b = 0; b < B && !any; ++b) any = run[b] && seqlens[b] > 0;
    if (!any) return L;
    std::vector<NormSeg> segs;
    int32_t prefix = 0, gprefix = 0;
    for (int32_t b = 0; b < B; ++b) {
      const int32_t S = seqlens[b];
      int32_t flags = 0;
      if (pending[b] && pending_split > 1) flags |= NORM_ADD_PARTIALS;
      if (run[b]) flags |= NORM_WRITE_OUT;
      if (!flags || S == 0) continue;
      NormSeg s{};
      s.row0 = cu[b]; s.prow0 = pcu[b]; s.nrows = S; s.prefix = prefix; s.flags = flags;
      s.gprefix = gprefix;
      segs.push_back(s);
      prefix += S;
      gprefix += (S + 7) / 8;
      L.write_out = L.write_out || run[b];
    }
    L.segs_off = w.append(segs);
    L.nsegs = (int32_t)segs.size();
    L.nrows = prefix;
    L.ngroups8 = gprefix;
    L.rows8 = rows8_ok && !rowvec && prefix > 0 && prefix >= rows8_min;
    L.nsplit = pending_split > 1 ? pending_split : 0;
    std::fill(pending.begin(), pending.end(), 0);
    pending_split = 0;
    return L;
  };

  std::vector<uint8_t> kv_on(KV), run_attn(B), run_ffn(B);
  for (int32_t l = 0; l < nlayers; ++l) {
    const LayerMasks& m = masks[l];
    LayerPlan& LP = plan->layers[l];
    std::vector<KChunk> chunks;
    push_chunks(chunks, 0, D, bk);   // dense K of the QKV and gate/up GEMMs
    const int32_t dense_cnt = (int32_t)chunks.size();

    GemmBuild qkv, o, gu, down;       // float32 path
    MmBuild mqkv, mo, mgu, mdown;     // 16-bit MFMA path
    std::vector<AttnGroup> ag;
    std::vector<int32_t> heads, kvheads;
    int32_t attn_tiles = 0, max_kv_cnt = 0;
    for (int32_t b = 0; b < B; ++b) {
      run_attn[b] = run_ffn[b] = 0;
      const int32_t S = seqlens[b];
      if (!m.layer_on[b] || S == 0) continue;
      const uint8_t* hm = m.head_mask + b * m.head_stride;
      const uint8_t* fm = m.ffn_mask ? m.ffn_mask + b * m.ffn_stride : nullptr;
      int32_t nh = 0;
      for (int32_t h = 0; h < A; ++h) nh += hm[h] ? 1 : 0;
      int32_t nf = 0;
      if (fm) { for (int32_t j = 0; j < G; ++j) nf += fm[j] ? 1 : 0; } else { nf = G; }
      if (nh > 0) {
        run_attn[b] = 1;
        for (int32_t g = 0; g < KV; ++g) {
          kv_on[g] = 0;
          for (int32_t h = g * rep; h < (g + 1) * rep; ++h) kv_on[g] |= hm[h];
        }
        // (section, weight matrix, active-head mask, heads, first output column)
        struct Sec { int32_t wsel; const uint8_t* on; int32_t n, col0; };
        const Sec secs[3] = {{0, hm, A, 0}, {1, kv_on.data(), KV, A * d},
                             {2, kv_on.data(), KV, (A + KV) * d}};
        for (const Sec& sc : secs)
          for (auto r : runs(sc.on, sc.n, d, 0)) {
            if (span) break;
            if (mfma)
              mqkv.add(pcu[b], pcu[b], S, sc.wsel, r.a, sc.col0 + r.a, (r.b - r.a) / 16, 0,
                       dense_cnt, sc.wsel < 2 ? 1 : 0, chunks, pos_base ? pos_base[b] : 0);
            else
              qkv.add(pcu[b], pcu[b], S, sc.col0 + r.a, sc.col0 + r.b, 0, dense_cnt);
          }
        // output projection: K runs over the active heads' columns of W_o
        int32_t off = (int32_t)chunks.size();
        for (auto r : runs(hm, A, d, 0)) push_chunks(chunks, r.a, r.b, bk);
        if (mfma)
          mo.add(pcu[b], cu[b], S, 0, 0, 0, D / 16, off, (int32_t)chunks.size() - off, 0, chunks);
        else
          o.add(pcu[b], cu[b], S, 0, D, off, (int32_t)chunks.size() - off);
        // attention: one group per sample
        AttnGroup g{};
        g.row0 = pcu[b]; g.S = S; g.h_off = (int32_t)heads.size(); g.h_cnt = nh;
        g.nqt = cdiv(S, ATTN_BQ); g.tile0 = attn_tiles;
        g.sample = b; g.pos_base = pos_base ? pos_base[b] : 0;
        g.kv_off = (int32_t)kvheads.size();
        for (int32_t h = 0; h < A; ++h) if (hm[h]) heads.push_back(h);
        for (int32_t k = 0; k < KV; ++k) if (kv_on[k]) kvheads.push_back(k);
        g.kv_cnt = (int32_t)kvheads.size() - g.kv_off;
        max_kv_cnt = std::max(max_kv_cnt, g.kv_cnt);
        attn_tiles += g.nqt * nh;
        ag.push_back(g);
      }
      if (nf > 0) {
        run_ffn[b] = 1;
        std::vector<uint8_t> all(G, 1);
        const uint8_t* fmm = fm ? fm : all.data();
        for (auto r : runs(fmm, G, slice, 0)) {
          if (span) break;
          if (mfma)
            mgu.add(pcu[b], pcu[b], S, 0, r.a, r.a, (r.b - r.a) / 8, 0, dense_cnt, 0, chunks);
          else
            gu.add(pcu[b], pcu[b], S, r.a, r.b, 0, dense_cnt);
        }
        int32_t off = (int32_t)chunks.size();
        for (auto r : runs(fmm, G, slice, 0)) push_chunks(chunks, r.a, r.b, bk);
        if (mfma)
          mdown.add(pcu[b], cu[b], S, 0, 0, 0, D / 16, off, (int32_t)chunks.size() - off, 0, chunks);
        else
          down.add(pcu[b], cu[b], S, 0, D, off, (int32_t)chunks.size() - off);
      }
    }

    if (span) {
      // rows [pcu[b0], last row of b1 - 1] of a run of consecutive samples
      auto run_rows = [&](int32_t b0, int32_t b1) { return pcu[b1 - 1] + seqlens[b1 - 1] - pcu[b0]; };
      using Runs = std::vector<std::pair<int32_t, int32_t>>;
      // the maximal runs of consecutive samples for which on(b) holds
      auto sample_runs = [&](auto on) {
        Runs r;
        for (int32_t b = 0; b < B;) {
          if (!on(b)) { ++b; continue; }
          const int32_t b0 = b;
          while (b < B && on(b)) ++b;
          r.push_back({b0, b});
        }
        return r;
      };
      // units u0 .. u1-1 (heads or FFN slices) with the same sample runs form
      // one group per run: emit(u0, u1, b0, b1)
      auto merged = [&](int32_t n, auto runs_of, auto emit) {
        int32_t u0 = 0;
        Runs cur = runs_of(0);
        for (int32_t u = 1; u <= n; ++u) {
          Runs nx = u < n ? runs_of(u) : Runs{};
          if (u < n && nx == cur) continue;
          for (const auto& r : cur) emit(u0, u, r.first, r.second);
          u0 = u;
          cur = std::move(nx);
        }
      };
      // QKV: heads (query, K/V) used by runs of samples
      struct SecS { int32_t wsel, n, col0; bool kv; };
      const SecS secs2[3] = {{0, A, 0, false}, {1, KV, A * d, true}, {2, KV, (A + KV) * d, true}};
      for (const SecS& sc : secs2)
        merged(sc.n,
               [&](int32_t h) {
                 return sample_runs([&](int32_t b) {
                   if (!run_attn[b]) return false;
                   const uint8_t* hm = m.head_mask + b * m.head_stride;
                   if (!sc.kv) return hm[h] != 0;
                   for (int32_t q = h * rep; q < (h + 1) * rep; ++q) if (hm[q]) return true;
                   return false;
                 });
               },
               [&](int32_t h0, int32_t h1, int32_t b0, int32_t b1) {
                 mqkv.add(pcu[b0], pcu[b0], run_rows(b0, b1), sc.wsel, h0 * d, sc.col0 + h0 * d,
                          (h1 - h0) * (d / 16), 0, dense_cnt, sc.wsel < 2 ? 1 : 0, chunks,
                          b1 - b0 > 1 ? -1 : 0);
               });
      // gate/up: FFN slices used by runs of samples
      merged(G,
             [&](int32_t j) {
               return sample_runs([&](int32_t b) {
                 return run_ffn[b] && (!m.ffn_mask || m.ffn_mask[b * m.ffn_stride + j]);
               });
             },
             [&](int32_t j0, int32_t j1, int32_t b0, int32_t b1) {
               mgu.add(pcu[b0], pcu[b0], run_rows(b0, b1), 0, j0 * slice, j0 * slice,
                       (j1 - j0) * slice / 8, 0, dense_cnt, 0, chunks);
             });
    }

    // attention sub-block
    LP.norm_attn = norm_launch(run_attn);
    if (mfma) {
      LP.qkv = mqkv.finish_paired(w, qkv_width, cap, plan->padded_rows, 2, force_split);
      LP.o = mo.finish_plain(w, R, D, cap, rowvec);
      const int32_t so = LP.o.nsplit;
      if (so > 1) {
        for (int32_t b = 0; b < B; ++b) pending[b] = run_attn[b];
        pending_split = so;
      }
    } else {
      LP.qkv = qkv.finish(w, BM, F32_BN, F32_BN, 1);
      LP.o = o.finish(w, BM, F32_BN, F32_BN, 1);
    }
    // 16-bit prefill attention: 32-row query tiles when 64-row tiles would
    // leave CUs idle (each workgroup then also splits its key range four
    // ways instead of two, so the longest tile's critical path halves)
    if (mfma && !rowvec && attn_tiles < kTargetTiles) {
      attn_tiles = 0;
      for (AttnGroup& g : ag) {
        g.nqt = cdiv(g.S, ATTN_BQ_SHORT);
        g.tile0 = attn_tiles;
        attn_tiles += g.nqt * g.h_cnt;
      }
      LP.attn.bq = ATTN_BQ_SHORT;
    }
    LP.attn.groups_off = w.append(ag);
    LP.attn.heads_off = w.append(heads);
    LP.attn.kvheads_off = w.append(kvheads);
    LP.attn.ngroups = (int32_t)ag.size();
    LP.attn.ntiles = attn_tiles;
    LP.attn.max_kv_cnt = max_kv_cnt;

    // FFN sub-block
    LP.norm_ffn = norm_launch(run_ffn);
    if (mfma) {
      LP.gu = mgu.finish_paired(w, 2 * F, cap, plan->padded_rows, 1, force_split);
      LP.down = mdown.finish_plain(w, R, D, cap, rowvec);
      const int32_t sd = LP.down.nsplit;
      if (sd > 1) {
        for (int32_t b = 0; b < B; ++b) pending[b] = run_ffn[b];
        pending_split = sd;
      }
    } else {
      LP.gu = gu.finish(w, BM, F32_SWIGLU_CH, F32_BN, 1);
      LP.down = down.finish(w, BM, F32_BN, F32_BN, 1);
    }
    if (mfma && rowvec && B > 1) {
      // decode of a batch: each weight block once for every sample using it
      DecBuild dq, dout, dgu, ddown;
      std::vector<uint8_t> on_h((size_t)B * std::max(A, KV));
      struct Sec { int32_t wsel, n, col0; bool kv; };
      const Sec secs[3] = {{0, A, 0, false}, {1, KV, A * d, true}, {2, KV, (A + KV) * d, true}};
      for (const Sec& sc : secs) {
        for (int32_t b = 0; b < B; ++b) {
          const uint8_t* hm = m.head_mask + b * m.head_stride;
          for (int32_t h = 0; h < sc.n; ++h) {
            uint8_t v = 0;
            if (run_attn[b]) {
              if (!sc.kv) v = hm[h];
              else for (int32_t q = h * rep; q < (h + 1) * rep; ++q) v |= hm[q];
            }
            on_h[(size_t)b * sc.n + h] = v;
          }
        }
        // runs of consecutive heads used by the same samples
        int32_t h0 = 0;
        while (h0 < sc.n) {
          std::vector<int32_t> smp;
          for (int32_t b = 0; b < B; ++b) if (on_h[(size_t)b * sc.n + h0]) smp.push_back(b);
          int32_t h1 = h0 + 1;
          while (h1 < sc.n) {
            bool same = true;
            for (int32_t b = 0; b < B && same; ++b)
              same = on_h[(size_t)b * sc.n + h1] == on_h[(size_t)b * sc.n + h0];
            if (!same) break;
            ++h1;
          }
          if (!smp.empty())
            dq.add((h1 - h0) * (d / 16), sc.wsel, h0 * d, sc.col0 + h0 * d, sc.wsel < 2 ? 1 : 0, smp,
                   pcu, pcu, pos_base, 0, dense_cnt, 0);
          h0 = h1;
        }
      }
      // FFN slices
      {
        std::vector<uint8_t> on_j((size_t)B * G);
        for (int32_t b = 0; b < B; ++b) {
          const uint8_t* fm = m.ffn_mask ? m.ffn_mask + b * m.ffn_stride : nullptr;
          for (int32_t j = 0; j < G; ++j) on_j[(size_t)b * G + j] = run_ffn[b] && (!fm || fm[j]);
        }
        int32_t j0 = 0;
        while (j0 < G) {
          std::vector<int32_t> smp;
          for (int32_t b = 0; b < B; ++b) if (on_j[(size_t)b * G + j0]) smp.push_back(b);
          int32_t j1 = j0 + 1;
          while (j1 < G) {
            bool same = true;
            for (int32_t b = 0; b < B && same; ++b) same = on_j[(size_t)b * G + j1] == on_j[(size_t)b * G + j0];
            if (!same) break;
            ++j1;
          }
          if (!smp.empty())
            dgu.add((j1 - j0) * slice / 8, 0, j0 * slice, j0 * slice, 0, smp, pcu, pcu, nullptr, 0,
                    dense_cnt, 0);
          j0 = j1;
        }
        // down projection: the union of the samples' active slices' chunks
        const int32_t fc = F / bk;
        std::vector<int32_t> chon((size_t)B * fc, 0);
        std::vector<int32_t> smp;
        for (int32_t b = 0; b < B; ++b) {
          if (!run_ffn[b]) continue;
          smp.push_back(b);
          for (int32_t c = 0; c < fc; ++c) chon[(size_t)b * fc + c] = on_j[(size_t)b * G + (c * bk) / slice];
        }
        if (!smp.empty())
          ddown.add(D / 16, 0, 0, 0, 0, smp, pcu, cu, nullptr, 0, 0, -1, &chon, fc, &chunks);
      }
      // output projection: the union of the samples' active heads' chunks
      {
        const int32_t oc = A * d / bk;
        std::vector<int32_t> chon((size_t)B * oc, 0);
        std::vector<int32_t> smp;
        for (int32_t b = 0; b < B; ++b) {
          if (!run_attn[b]) continue;
          smp.push_back(b);
          const uint8_t* hm = m.head_mask + b * m.head_stride;
          for (int32_t c = 0; c < oc; ++c) chon[(size_t)b * oc + c] = hm[(c * bk) / d];
        }
        if (!smp.empty())
          dout.add(D / 16, 0, 0, 0, 0, smp, pcu, cu, nullptr, 0, 0, -1, &chon, oc, &chunks);
      }
      dq.finish(w, LP.qkv);
      dout.finish(w, LP.o);
      dgu.finish(w, LP.gu);
      ddown.finish(w, LP.down);
    }
    LP.chunks_off = w.append(chunks);
  }
  std::vector<uint8_t> none(B, 0);
  plan->final_norm = norm_launch(none, true);
  return true;
}

}  // namespace svl
