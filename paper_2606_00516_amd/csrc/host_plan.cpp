#include "host_plan.h"

#include <algorithm>
#include <numeric>

namespace eb {

namespace {
constexpr int kPagesPerSplit = 32;  // must match kDecodePagesPerSplit
constexpr int kPage = 16;
constexpr int kShortKeys = 64;      // must match kShortDecodeKeys
constexpr int kShortHeads = 4;      // must match kShortDecodeHeads

// query positions per prefill item (must match the attention kernels)
int prefill_bq_host(int group, bool mixed_launch) {
  return mixed_launch ? 128 / group : 128 / group;
}
}  // namespace

int32_t decode_splits(int32_t c) {
  const int32_t keys = c + 1;
  const int32_t per = kPagesPerSplit * kPage;
  return (keys + per - 1) / per;
}

eb_status check_config(const eb_layer_config *cfg, std::string &err) {
  if (!cfg) {
    err = "config is NULL";
    return EB_ERR_NULL;
  }
  const eb_layer_config &c = *cfg;
  if (c.hidden <= 0 || c.n_q_heads <= 0 || c.n_kv_heads <= 0 || c.head_dim <= 0 || c.ffn < 0 ||
      (c.ffn == 0 && c.n_experts <= 0)) {
    err = "layer sizes must be positive";
    return EB_ERR_CONFIG;
  }
  if (c.head_dim != 64 && c.head_dim != 128) {
    err = "head_dim must be 64 or 128";
    return EB_ERR_CONFIG;
  }
  if (c.n_q_heads % c.n_kv_heads != 0) {
    err = "n_q_heads must be a multiple of n_kv_heads";
    return EB_ERR_CONFIG;
  }
  const int g = c.n_q_heads / c.n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) {
    err = "n_q_heads / n_kv_heads must be 1, 2, 4 or 8";
    return EB_ERR_CONFIG;
  }
  if (c.page_size != kPage) {
    err = "page_size must be 16";
    return EB_ERR_CONFIG;
  }
  if (c.hidden % 8 || c.ffn % 8) {
    err = "hidden and ffn must be multiples of 8";
    return EB_ERR_CONFIG;
  }
  if (c.n_experts < 0) {
    err = "n_experts must be >= 0";
    return EB_ERR_CONFIG;
  }
  if (c.n_experts > 0) {
    if (c.n_experts % 16 || c.n_experts > 256 || c.top_k < 1 || c.top_k > c.n_experts || c.top_k > 64 ||
        c.expert_ffn <= 0 || c.expert_ffn % 8 || c.hidden % 32) {
      err = "mixture-of-experts layer: n_experts a multiple of 16 up to 256, 1 <= top_k <= min(n_experts, 64), "
            "expert_ffn a positive multiple of 8, hidden a multiple of 32";
      return EB_ERR_CONFIG;
    }
  }
  if (!(c.rms_eps > 0.f) || !(c.rope_theta > 0.f)) {
    err = "rms_eps and rope_theta must be positive";
    return EB_ERR_CONFIG;
  }
  return EB_OK;
}

eb_status check_batch(const eb_layer_config &cfg, const eb_batch *b, int32_t max_pages_per_seq, eb_mode mode,
                      std::string &err) {
  if (!b) {
    err = "batch is NULL";
    return EB_ERR_NULL;
  }
  if (mode != EB_MODE_DECODE && mode != EB_MODE_PREFILL && mode != EB_MODE_MIXED) {
    err = "unknown mode";
    return EB_ERR_MODE;
  }
  if (b->num_seqs < 0 || b->num_tokens < 0) {
    err = "negative num_seqs or num_tokens";
    return EB_ERR_BATCH;
  }
  if (b->num_seqs == 0) {
    if (b->num_tokens != 0) {
      err = "num_tokens must be 0 for an empty batch";
      return EB_ERR_BATCH;
    }
    return EB_OK;
  }
  if (!b->context_lens_host || !b->chunk_lens_host) {
    err = "context_lens_host / chunk_lens_host is NULL";
    return EB_ERR_NULL;
  }
  int64_t sum = 0;
  for (int i = 0; i < b->num_seqs; ++i) {
    const int32_t c = b->context_lens_host[i], n = b->chunk_lens_host[i];
    if (n < 1) {
      err = "request " + std::to_string(i) + ": chunk_len must be >= 1";
      return EB_ERR_BATCH;
    }
    if (c < 0) {
      err = "request " + std::to_string(i) + ": negative context_len";
      return EB_ERR_BATCH;
    }
    if (mode == EB_MODE_DECODE && n != 1) {
      err = "decode mode: request " + std::to_string(i) + " has chunk_len " + std::to_string(n);
      return EB_ERR_MODE;
    }
    if ((int64_t)c + n > (int64_t)0x3FFFFFFF) {
      err = "request " + std::to_string(i) + ": length overflows";
      return EB_ERR_BATCH;
    }
    if (max_pages_per_seq >= 0 && (int64_t)c + n > (int64_t)max_pages_per_seq * cfg.page_size) {
      err = "request " + std::to_string(i) + ": context + chunk exceeds max_pages_per_seq * page_size";
      return EB_ERR_PAGES;
    }
    sum += n;
  }
  if (sum != b->num_tokens) {
    err = "num_tokens (" + std::to_string(b->num_tokens) + ") != sum of chunk_lens (" + std::to_string(sum) + ")";
    return EB_ERR_BATCH;
  }
  return EB_OK;
}

eb_status check_tables(const eb_layer_config &cfg, const eb_batch &b, const int32_t *bt, int32_t num_pages,
                       int32_t max_pages_per_seq, std::string &err) {
  if (b.num_seqs == 0) return EB_OK;
  if (!bt) {
    err = "block_tables_host is NULL";
    return EB_ERR_NULL;
  }
  if (num_pages <= 0 || max_pages_per_seq <= 0) {
    err = "num_pages and max_pages_per_seq must be positive";
    return EB_ERR_PAGES;
  }
  std::vector<int32_t> owner((size_t)num_pages, -1);
  for (int i = 0; i < b.num_seqs; ++i) {
    const int64_t need = ((int64_t)b.context_lens_host[i] + b.chunk_lens_host[i] + cfg.page_size - 1) / cfg.page_size;
    for (int64_t j = 0; j < need; ++j) {
      const int32_t id = bt[(size_t)i * max_pages_per_seq + j];
      if (id < 0 || id >= num_pages) {
        err = "request " + std::to_string(i) + " logical page " + std::to_string(j) + ": id " + std::to_string(id) +
              " outside [0, num_pages)";
        return EB_ERR_PAGES;
      }
      if (owner[id] >= 0) {
        err = "physical page " + std::to_string(id) + " is used twice";
        return EB_ERR_PAGES;
      }
      owner[id] = i;
    }
  }
  return EB_OK;
}

size_t plan_capacity(int32_t max_seqs, int32_t max_tokens, int32_t group) {
  const size_t S = (size_t)max_seqs, T = (size_t)max_tokens;
  const size_t tiles = T / (size_t)std::min(prefill_bq_host(group, true), prefill_bq_host(group, false)) + S + 1;
  return 6 * S + kDecInfo * (S + 1) + kCombInfo * S + 2 * T + 2 * tiles + 64;  // + per-array alignment padding
}

void build_plan(const eb_layer_config &cfg, const eb_batch &b, eb_mode mode, HostPlan &p) {
  const int S = b.num_seqs, T = b.num_tokens;
  bool any_dec = false, any_pf = false;
  for (int i = 0; i < S; ++i) (b.chunk_lens_host[i] == 1 ? any_dec : any_pf) = true;
  const bool mixed_launch = mode == EB_MODE_MIXED && any_dec && any_pf;
  const int bq = prefill_bq_host(cfg.n_q_heads / cfg.n_kv_heads, mixed_launch);
  p = HostPlan();
  p.S = S;
  p.T = T;
  std::vector<int32_t> row(S + 1, 0), goff(S + 1, 0);
  for (int i = 0; i < S; ++i) {
    row[i + 1] = row[i] + b.chunk_lens_host[i];
    goff[i + 1] = goff[i] + b.context_lens_host[i] + b.chunk_lens_host[i];
  }
  p.gather_total = goff[S];
  std::vector<int32_t> row_seq(T), row_pos(T), dec_seq, dec_off(1, 0), full_off(1, 0), comb, shorts;
  struct Part {
    int32_t d, pages;
  };
  std::vector<Part> parts;
  const int nkv = cfg.n_kv_heads;
  struct Tile {
    int32_t seq, qb, cost;
  };
  std::vector<Tile> tiles;
  for (int i = 0; i < S; ++i) {
    const int32_t c = b.context_lens_host[i], n = b.chunk_lens_host[i];
    for (int j = 0; j < n; ++j) {
      row_seq[row[i] + j] = i;
      row_pos[row[i] + j] = c + j;
    }
    if (n == 1) {
      const int32_t ns = decode_splits(c);
      const int32_t d = (int32_t)dec_seq.size();
      if (ns >= 2) comb.push_back(d);
      dec_seq.push_back(i);
      dec_off.push_back(dec_off.back() + ns);
      const int32_t keys = c + 1, per = kPagesPerSplit * kPage;
      int32_t nfull = 0;
      if (keys <= kShortKeys) {
        shorts.push_back(d);
      } else {
        nfull = keys / per;  // splits of exactly 32 pages
        if (keys % per) parts.push_back({d, (keys % per + kPage - 1) / kPage});
      }
      full_off.push_back(full_off.back() + nfull * nkv);
    } else {
      const int nqb = (n + bq - 1) / bq;
      for (int qb = 0; qb < nqb; ++qb) tiles.push_back({i, qb, c + std::min(n, (qb + 1) * bq)});
    }
  }
  std::stable_sort(tiles.begin(), tiles.end(), [](const Tile &a, const Tile &b) { return a.cost > b.cost; });
  // longest last splits first (ties in request order): the launch ends on
  // the shortest units, which keeps its tail short
  std::stable_sort(parts.begin(), parts.end(), [](const Part &a, const Part &b) { return a.pages > b.pages; });
  p.n_dec = (int32_t)dec_seq.size();
  p.total_splits = dec_off.back();
  p.n_full_units = full_off.back();
  p.n_part = (int32_t)parts.size();
  p.n_short = (int32_t)shorts.size();
  p.total_units = p.n_full_units + p.n_part * nkv + p.n_short * ((nkv + kShortHeads - 1) / kShortHeads);
  p.n_comb = (int32_t)comb.size();
  p.n_tiles = (int32_t)tiles.size();

  auto &B = p.blob;
  auto put = [&](const int32_t *src, size_t n) {
    const size_t off = B.size();
    B.insert(B.end(), src, src + n);
    // keep every array 16-byte aligned
    while (B.size() % 4) B.push_back(0);
    return off;
  };
  p.o_ctx = put(b.context_lens_host, (size_t)S);
  p.o_len = put(b.chunk_lens_host, (size_t)S);
  p.o_row = put(row.data(), row.size());
  p.o_row_seq = put(row_seq.data(), row_seq.size());
  p.o_row_pos = put(row_pos.data(), row_pos.size());
  // one record per decode request and a closing one (totals)
  std::vector<int32_t> info((size_t)kDecInfo * (dec_seq.size() + 1), 0);
  for (size_t d = 0; d <= dec_seq.size(); ++d) {
    int32_t *r = &info[d * kDecInfo];
    r[0] = full_off[d];
    r[1] = dec_off[d];
    if (d < dec_seq.size()) {
      const int i = dec_seq[d];
      r[2] = i;
      r[3] = row[i];
      r[4] = b.context_lens_host[i] + 1;
      r[5] = dec_off[d + 1] - dec_off[d];
    }
  }
  p.o_dec_info = put(info.data(), info.size());
  std::vector<int32_t> part_d(parts.size());
  for (size_t j = 0; j < parts.size(); ++j) part_d[j] = parts[j].d;
  p.o_part = put(part_d.data(), part_d.size());
  p.o_short = put(shorts.data(), shorts.size());
  std::vector<int32_t> comb_rec((size_t)kCombInfo * comb.size(), 0);
  for (size_t j = 0; j < comb.size(); ++j) {
    const int d = comb[j];
    comb_rec[j * kCombInfo + 0] = dec_off[d];
    comb_rec[j * kCombInfo + 1] = dec_off[d + 1] - dec_off[d];
    comb_rec[j * kCombInfo + 2] = row[dec_seq[d]];
  }
  p.o_comb = put(comb_rec.data(), comb_rec.size());
  std::vector<int32_t> tseq(tiles.size()), tqb(tiles.size());
  for (size_t t = 0; t < tiles.size(); ++t) {
    tseq[t] = tiles[t].seq;
    tqb[t] = tiles[t].qb;
  }
  p.o_tseq = put(tseq.data(), tseq.size());
  p.o_tqb = put(tqb.data(), tqb.size());
  p.o_goff = put(goff.data(), goff.size());
  if (B.empty()) B.assign(4, 0);
}

}  // namespace eb
