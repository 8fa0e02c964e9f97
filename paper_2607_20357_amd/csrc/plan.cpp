// Host planner.  For each layer it lists, per executed sample:
//   * the packed rows that run the attention / FFN sub-blocks (norm runs);
//   * the active output-column ranges of the QKV and gate/up GEMMs (only
//     active heads' and active FFN slices' weight rows are ever read);
//   * the active K chunks of the output and down projections (only active
//     heads' / slices' weight columns are ever read);
//   * the active heads of the attention launch.
// It also picks the bf16 GEMM tile width of each launch: narrow tiles for
// skinny samples, so that a launch has enough workgroups for the 256 CUs
// without splitting K.
#include "plan.h"

#include <algorithm>
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
  int32_t max_rows = 0;
  void add(int32_t row0, int32_t nrows, int32_t n0, int32_t n1, int32_t kc_off, int32_t kc_cnt) {
    if (nrows <= 0 || n1 <= n0 || kc_cnt <= 0) return;
    GemmGroup g{};
    g.row0 = row0; g.nrows = nrows; g.n0 = n0; g.n1 = n1;
    g.kc_off = kc_off; g.kc_cnt = kc_cnt;
    groups.push_back(g);
    max_rows = std::max(max_rows, nrows);
  }
  // Numbers the tiles (M tile fastest) for tiles of BM rows x BNO output
  // columns; bn is the tile width in weight rows recorded for the launch.
  GemmLaunch finish(ImageWriter& w, int32_t BM, int32_t BNO, int32_t bn) {
    GemmLaunch L;
    int32_t tile = 0;
    for (auto& g : groups) {
      g.tile0 = tile;
      tile += cdiv(g.nrows, BM) * cdiv(g.n1 - g.n0, BNO);
    }
    L.groups_off = w.append(groups);
    L.ngroups = (int32_t)groups.size();
    L.ntiles = tile;
    L.bn = bn;
    return L;
  }
};

// K chunks covering [a, b) in pieces of at most `bk` columns.
void push_chunks(std::vector<KChunk>& ch, int32_t a, int32_t b, int32_t bk) {
  for (int32_t k = a; k < b; k += bk) ch.push_back({k, std::min(bk, b - k)});
}

}  // namespace

int64_t plan_bytes_bound(const svl_config& c, int32_t B, int32_t nlayers) {
  const int64_t A = c.n_heads, KV = c.n_kv_heads, G = c.n_groups, d = c.head_dim;
  const int64_t F = c.d_ffn, D = c.d_model;
  const int64_t bk = 64;
  int64_t per_layer = 0;
  per_layer += 2 * (B * (int64_t)sizeof(Seg) + 16);
  // QKV: at most one range per head (q) and per kv head (k and v)
  per_layer += B * (A + 2 * KV) * (int64_t)sizeof(GemmGroup) + 16;
  per_layer += B * (int64_t)sizeof(GemmGroup) + 16;                 // o
  per_layer += B * G * (int64_t)sizeof(GemmGroup) + 16;             // gate/up
  per_layer += B * (int64_t)sizeof(GemmGroup) + 16;                 // down
  per_layer += B * (int64_t)sizeof(AttnGroup) + 16;
  per_layer += B * A * 4 + 16;
  // chunks: dense D, per sample active head columns and FFN slices
  int64_t chunks = (D + bk - 1) / bk + B * A * ((d + bk - 1) / bk) +
                   B * G * ((F / G + bk - 1) / bk);
  per_layer += chunks * (int64_t)sizeof(KChunk) + 16;
  return 64 + (int64_t)B * 4 + (int64_t)(B + 1) * 4 + 32 + per_layer * nlayers;
}

bool build_plan(const svl_config& cfg, int32_t B, const int32_t* keep, const int32_t* seqlens,
                int32_t nlayers, const LayerMasks* masks, Plan* plan, std::string* err) {
  const bool bf16 = cfg.dtype == SVL_BF16;
  const int32_t A = cfg.n_heads, KV = cfg.n_kv_heads, G = cfg.n_groups, d = cfg.head_dim;
  const int32_t D = cfg.d_model, F = cfg.d_ffn, rep = A / KV, slice = F / G;
  const int32_t BM = bf16 ? BF16_BM : F32_BM;
  const int32_t bk = 64;

  plan->image.clear();
  plan->layers.assign(nlayers, LayerPlan{});
  plan->max_seq = 0;
  ImageWriter w{&plan->image};

  std::vector<int32_t> cu(B + 1, 0);
  for (int32_t b = 0; b < B; ++b) {
    if (seqlens[b] < 0) { *err = "negative sequence length"; return false; }
    cu[b + 1] = cu[b] + seqlens[b];
    plan->max_seq = std::max(plan->max_seq, seqlens[b]);
  }
  std::vector<int32_t> kp(B, 0);
  if (keep) for (int32_t b = 0; b < B; ++b) kp[b] = keep[b];
  plan->keep_off = w.append(kp);
  plan->cu_off = w.append(cu);

  std::vector<uint8_t> kv_on(KV);
  for (int32_t l = 0; l < nlayers; ++l) {
    const LayerMasks& m = masks[l];
    LayerPlan& LP = plan->layers[l];
    std::vector<KChunk> chunks;
    push_chunks(chunks, 0, D, bk);   // dense K of the QKV and gate/up GEMMs
    const int32_t dense_cnt = (int32_t)chunks.size();

    std::vector<Seg> seg_a, seg_f;
    GemmBuild qkv, o, gu, down;
    std::vector<AttnGroup> ag;
    std::vector<int32_t> heads;
    int32_t attn_tiles = 0;
    for (int32_t b = 0; b < B; ++b) {
      const int32_t S = seqlens[b];
      if (!m.layer_on[b] || S == 0) continue;
      const uint8_t* hm = m.head_mask + b * m.head_stride;
      const uint8_t* fm = m.ffn_mask ? m.ffn_mask + b * m.ffn_stride : nullptr;
      int32_t nh = 0;
      for (int32_t h = 0; h < A; ++h) nh += hm[h] ? 1 : 0;
      int32_t nf = 0;
      if (fm) { for (int32_t j = 0; j < G; ++j) nf += fm[j] ? 1 : 0; } else { nf = G; }
      const int32_t row0 = cu[b];
      if (nh > 0) {
        int32_t prefix = seg_a.empty() ? 0 : seg_a.back().prefix + seg_a.back().nrows;
        seg_a.push_back({row0, S, prefix, 0});
        for (auto r : runs(hm, A, d, 0)) qkv.add(row0, S, r.a, r.b, 0, dense_cnt);
        for (int32_t g = 0; g < KV; ++g) {
          kv_on[g] = 0;
          for (int32_t h = g * rep; h < (g + 1) * rep; ++h) kv_on[g] |= hm[h];
        }
        for (auto r : runs(kv_on.data(), KV, d, A * d)) qkv.add(row0, S, r.a, r.b, 0, dense_cnt);
        for (auto r : runs(kv_on.data(), KV, d, (A + KV) * d))
          qkv.add(row0, S, r.a, r.b, 0, dense_cnt);
        // output projection: K runs over the active heads' columns of W_o
        int32_t off = (int32_t)chunks.size();
        for (auto r : runs(hm, A, d, 0)) push_chunks(chunks, r.a, r.b, bk);
        o.add(row0, S, 0, D, off, (int32_t)chunks.size() - off);
        // attention: one group per sample
        AttnGroup g{};
        g.row0 = row0; g.S = S; g.h_off = (int32_t)heads.size(); g.h_cnt = nh;
        g.nqt = cdiv(S, ATTN_BQ); g.tile0 = attn_tiles;
        for (int32_t h = 0; h < A; ++h) if (hm[h]) heads.push_back(h);
        attn_tiles += g.nqt * nh;
        ag.push_back(g);
      }
      if (nf > 0) {
        int32_t prefix = seg_f.empty() ? 0 : seg_f.back().prefix + seg_f.back().nrows;
        seg_f.push_back({row0, S, prefix, 0});
        std::vector<uint8_t> all(G, 1);
        const uint8_t* fmm = fm ? fm : all.data();
        for (auto r : runs(fmm, G, slice, 0)) gu.add(row0, S, r.a, r.b, 0, dense_cnt);
        int32_t off = (int32_t)chunks.size();
        for (auto r : runs(fmm, G, slice, 0)) push_chunks(chunks, r.a, r.b, bk);
        down.add(row0, S, 0, D, off, (int32_t)chunks.size() - off);
      }
    }
    auto seg_rows = [](const std::vector<Seg>& s) {
      return s.empty() ? 0 : s.back().prefix + s.back().nrows;
    };
    LP.norm_attn.segs_off = w.append(seg_a);
    LP.norm_attn.nsegs = (int32_t)seg_a.size();
    LP.norm_attn.nrows = seg_rows(seg_a);
    LP.norm_ffn.segs_off = w.append(seg_f);
    LP.norm_ffn.nsegs = (int32_t)seg_f.size();
    LP.norm_ffn.nrows = seg_rows(seg_f);
    if (bf16) {
      // narrow tiles for skinny samples: enough workgroups without split-K
      const int32_t bn_od = std::max(o.max_rows, down.max_rows) <= kSkinnyRows ? 32 : 64;
      const int32_t bn_gu = gu.max_rows <= kSkinnyRows ? 64 : 128;
      LP.qkv = qkv.finish(w, BM, 64, 64);
      LP.o = o.finish(w, BM, bn_od, bn_od);
      LP.gu = gu.finish(w, BM, bn_gu / 2, bn_gu);
      LP.down = down.finish(w, BM, bn_od, bn_od);
    } else {
      LP.qkv = qkv.finish(w, BM, F32_BN, F32_BN);
      LP.o = o.finish(w, BM, F32_BN, F32_BN);
      LP.gu = gu.finish(w, BM, F32_SWIGLU_CH, F32_BN);
      LP.down = down.finish(w, BM, F32_BN, F32_BN);
    }
    LP.attn.groups_off = w.append(ag);
    LP.attn.heads_off = w.append(heads);
    LP.attn.ngroups = (int32_t)ag.size();
    LP.attn.ntiles = attn_tiles;
    LP.chunks_off = w.append(chunks);
  }
  (void)bf16;
  return true;
}

}  // namespace svl
