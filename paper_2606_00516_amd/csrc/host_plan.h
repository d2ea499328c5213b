// Host-side validation and launch planning for one step.  Pure C++: no HIP
// calls, so it runs (and is tested) without a GPU.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/eb_layer.h"

namespace eb {

// int32 fields of a decode request's record: first work unit among the
// full splits, first split, request, first row, keys (c + 1), splits,
// padding to 32 bytes
constexpr int kDecInfo = 8;
// int32 fields of a combine record (decode request with >= 2 splits): first
// split, splits, row, padding
constexpr int kCombInfo = 4;

struct HostPlan {
  int32_t S = 0, T = 0;
  int32_t n_dec = 0, total_splits = 0, total_units = 0, n_comb = 0, n_tiles = 0;
  // decode work units in launch order: the full 32-page splits (request by
  // request, n_full_units of them), then the requests' shorter last splits,
  // longest first (n_part requests x n_kv units), then the requests of at
  // most kShortKeys keys (n_short of them)
  int32_t n_full_units = 0, n_part = 0, n_short = 0;
  int64_t gather_total = 0;
  std::vector<int32_t> blob;  // every metadata array, concatenated
  // offsets (in int32 elements) of each array inside blob
  size_t o_ctx = 0, o_len = 0, o_row = 0, o_row_seq = 0, o_row_pos = 0, o_dec_info = 0, o_comb = 0, o_tseq = 0,
         o_tqb = 0, o_goff = 0, o_part = 0, o_short = 0;
};

// Shape support: head_dim in {64, 128}; G = n_q / n_kv in {1, 2, 4, 8};
// page_size 16; hidden, ffn multiples of 8; positive sizes and eps, theta.
eb_status check_config(const eb_layer_config *cfg, std::string &err);

// Lengths and mode constraints.  max_pages_per_seq < 0 skips the capacity
// check (used where no cache is involved).
eb_status check_batch(const eb_layer_config &cfg, const eb_batch *b, int32_t max_pages_per_seq, eb_mode mode,
                      std::string &err);

// Block-table contents on the host: ids in [0, num_pages) for every needed
// logical page, and no physical page used twice.
eb_status check_tables(const eb_layer_config &cfg, const eb_batch &b, const int32_t *bt_host, int32_t num_pages,
                       int32_t max_pages_per_seq, std::string &err);

// Build the metadata of a step: row offsets, per-row request and position,
// the decode split list, the prefill tile list (longest first) and gather
// offsets.  The batch must have passed check_batch.
// The prefill item size depends on the launch: `mode` says which launch the
// step makes (a mixed batch in EB_MODE_MIXED uses the single mixed grid).
void build_plan(const eb_layer_config &cfg, const eb_batch &b, eb_mode mode, HostPlan &p);

// Upper bound of blob size (int32 elements) for a handle's limits.
size_t plan_capacity(int32_t max_seqs, int32_t max_tokens, int32_t group);

// Decode splits of a request with c cached tokens (it attends to c + 1 keys).
int32_t decode_splits(int32_t c);

}  // namespace eb
