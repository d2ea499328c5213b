// Internal interfaces between the host planner/launcher and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace eb {

// Decode attention splits a request's keys into fixed chunks of this many
// pages (tokens = pages * 16).  The count depends only on the request's own
// length, so its result is the same in any batch.
constexpr int kDecodePagesPerSplit = 32;
constexpr int kPageSize = 16;
// A decode request with at most this many keys (context + 1) runs as units
// of kShortDecodeHeads kv heads, one wavefront each, instead of page splits.
constexpr int kShortDecodeKeys = 64;
constexpr int kShortDecodeHeads = 4;
// int32 fields per decode-request record in DevMeta::dec_info
constexpr int kDecInfoInts = 8;
// int32 fields per record in DevMeta::comb_list
constexpr int kCombInfoInts = 4;

// Prefill attention items: query positions per item for a GQA group size,
// in the prefill-only launch and inside the mixed launch (must agree with
// PrefillTraits in the attention kernels).
inline int prefill_bq(int group, bool mixed_launch) {
  return mixed_launch ? 128 / group : 128 / group;
}

// Work order of the single mixed attention launch.  Its P prefill items are
// compute bound and its D decode units stream K/V from HBM; placing the
// prefill items at every s-th block over the first kMixedPrefillSpan of the
// grid (longest first) keeps both kinds running side by side on the CUs
// instead of one phase after the other.  Block b runs prefill item b / s
// when b % s == 0 and b / s < P, otherwise decode unit b - min(P, b / s + 1).
#ifndef EB_MIX_SPAN
#define EB_MIX_SPAN 80
#endif
constexpr int kMixedPrefillSpanPct = EB_MIX_SPAN;
inline int mixed_prefill_stride(long P, long D) {
  if (P <= 0 || D <= 0) return 1;
  const long s = (long)kMixedPrefillSpanPct * (P + D) / (100 * P);
  return s < 1 ? 1 : (s > (1L << 30) ? (1 << 30) : (int)s);
}

// Per-step metadata in device memory (all int32), produced by the planner.
struct DevMeta {
  const int32_t *seq_ctx;       // [S] tokens cached before the step
  const int32_t *seq_len;       // [S] new rows
  const int32_t *seq_row;       // [S+1] first row of each request
  const int32_t *row_seq;       // [T] request of each row
  const int32_t *row_pos;       // [T] absolute position of each row
  const int32_t *dec_info;      // [D+1][8] {first full-split unit, first split, request, row, keys, splits,
                                // 0, 0}; the closing record holds the full-split unit count
  const int32_t *dec_part;      // [n_part] requests whose last split is shorter, longest first
  const int32_t *dec_short;     // [n_short] requests of at most kShortDecodeKeys keys
  const int32_t *comb_list;     // [C][4] decode requests with >= 2 splits: {first split, splits, row, 0}
  const int32_t *tile_seq;      // [NT] prefill tiles, longest first
  const int32_t *tile_qb;       // [NT] query block of each tile
  const int32_t *gather_off;    // [S+1] prefix sum of (c + n)
  int32_t S, T, n_dec, total_splits, total_units, n_comb, n_tiles;
  int32_t n_full_units, n_part, n_short;  // decode units: full splits, then shorter last splits, then short requests
};

struct KV {
  uint16_t *k, *v;      // element type per f8: bf16, or 8-bit E4M3 codes (read through k8 / v8)
  const int32_t *bt;
  int32_t num_pages, max_pages;
  int32_t f8;           // 1: 8-bit codes
  float ks, vs;         // value of a code = decode(code) * scale (8-bit caches)
  __host__ __device__ uint8_t *k8() const { return reinterpret_cast<uint8_t *>(k); }
  __host__ __device__ uint8_t *v8() const { return reinterpret_cast<uint8_t *>(v); }
};

struct Shape {
  int32_t hidden, nq, nkv, hd, ffn;
  float eps, theta;
  int32_t ne = 0, topk = 0, effn = 0, renorm = 1;  // mixture-of-experts feed-forward when ne > 0
  int32_t qkn = 0;                                  // per-head q/k RMSNorm before RoPE
  bool moe() const { return ne > 0; }
  int32_t qkv_cols() const { return (nq + 2 * nkv) * hd; }
  int32_t group() const { return nq / nkv; }
};

// Fixed device scratch of the no-allocation step entry point: its size, and
// the device address of the calling device's copy (looked up once per
// device with that device current).
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
hipError_t noalloc_scratch_setup(int device, void **addr);

// ---- launchers (each returns the launch error) ----
hipError_t launch_rmsnorm(const uint16_t *x, const uint16_t *gamma, uint16_t *out, int rows, int d, float eps,
                          hipStream_t st);
// gq, gk: the per-head norm gains, required when s.qkn
hipError_t launch_rope_append(const Shape &s, uint16_t *qkv, const KV &kv, const DevMeta &m, hipStream_t st,
                              const uint16_t *gq = nullptr, const uint16_t *gk = nullptr);
// The RoPE/append of a decode-sized step fused with the QKV projection's
// split-K sum and the row scale of the RMSNorm before it: part holds the
// projection's fp32 partials [splits][T][qkv_cols] of x * g1, ssq the rows'
// partial sums of squares [splits][T] (launch_gemm_prenorm).
hipError_t launch_qkv_rope_append(const Shape &s, const float *part, int splits, const float *ssq, uint16_t *qkv,
                                  const KV &kv, const DevMeta &m, hipStream_t st, const uint16_t *gq = nullptr,
                                  const uint16_t *gk = nullptr);
hipError_t launch_gather_kv(const Shape &s, const KV &kv, const DevMeta &m, uint16_t *out_k, uint16_t *out_v,
                            hipStream_t st);

// attention: kind 0 = decode only, 1 = prefill only, 2 = mixed single launch;
// parts: 1 = the attention kernel(s), 2 = the decode split combine, 3 = both
hipError_t launch_attention(const Shape &s, const uint16_t *qkv, const KV &kv, const DevMeta &m, uint16_t *out,
                            float *part_o, float *part_ml, int kind, hipStream_t st, int parts = 3);

// GEMM planning shared by the op entry and the step.
enum GemmEpi { EPI_STORE = 0, EPI_RESIDUAL = 1, EPI_SILU_MUL = 2 };
struct GemmPlan {
  int kind;      // 0 = skinny weight-streaming, 1 = LDS-tiled, 2 = 256 x 256 tiles, -1 = none fits
  int splits;    // split-K factor (skinny, and big with few tiles)
  int kt_per;    // big: 64-wide K tiles per split
  size_t ws_bytes;
};
// w8: W holds 8-bit E4M3 codes with one fp32 scale per row (launch_gemm's
// wscale, null for bf16 weights); such plans never take the tiled kernel.
GemmPlan plan_gemm(int M, int N, int K, int epi, bool w8 = false);
// With nf, a residual GEMM whose plan splits K also writes the RMSNorm of
// its result rows (gamma, out, eps) from the split-K sum and sets nf->done;
// otherwise nf->done stays false and the caller runs the norm itself.
struct NormFuse {
  const uint16_t *gamma;
  uint16_t *out;
  float eps;
  bool done;
};
hipError_t launch_gemm(const GemmPlan &p, const uint16_t *A, const void *W, const float *wscale, uint16_t *out,
                       const uint16_t *residual, int M, int N, int K, int epi, void *ws, hipStream_t st,
                       NormFuse *nf = nullptr, const uint16_t *Wp = nullptr);
// Wp: optional fragment-packed copy of a bf16 W (pack_weight); the
// weight-streaming plans read it instead of W when packed_ok(N, K, epi).
bool packed_ok(int N, int K, int epi);
size_t packed_weight_bytes(int N, int K);
hipError_t pack_weight(const uint16_t *W, uint16_t *P, int N, int K, hipStream_t st);

// The weight-streaming GEMM on the RMSNorm that precedes it: stages bf16(x *
// gamma) as A and writes the split-K partials only (p.kind 0 with
// p.splits >= 2), plus each row's partial sum of squares of x into ssq
// [p.splits][M]; the consumer applies 1 / sqrt(mean(x^2) + eps) to the sum.
hipError_t launch_gemm_prenorm(const GemmPlan &p, const uint16_t *x, const uint16_t *gamma, const void *W,
                               const float *wscale, int M, int N, int K, float *part, float *ssq, hipStream_t st,
                               const uint16_t *Wp = nullptr);

// Mixture-of-experts block.  The grouped GEMM multiplies row tiles of
// expert-sorted rows (tables [3][max_tiles]: expert, first sorted row, rows;
// *n_tiles of them in use) by their expert's W ([E][N][K] bf16), gathering A
// rows through a_rows (null: the sorted row itself); SiLU epilogue to bf16
// [rows, N / 2], or store to fp32 [rows, N] when f32_out.
hipError_t launch_gemm_grouped(const uint16_t *A, int a_nrows, const int32_t *a_rows, const uint16_t *W, void *out,
                               bool f32_out, const int32_t *tiles, const int32_t *n_tiles, int max_tiles, int N, int K,
                               int epi, hipStream_t st);
// The same on the 256 x 256 kernel: tiles of up to 256 rows, K a multiple of 64.
hipError_t launch_gemm_grouped_big(const uint16_t *A, int a_nrows, const int32_t *a_rows, const uint16_t *W,
                                   void *out, bool f32_out, const int32_t *tiles, const int32_t *n_tiles, int max_tiles,
                                   int N, int K, int epi, hipStream_t st);
hipError_t launch_moe_route(const uint16_t *b, const uint16_t *wr, int T, int d, int E, int k, int renormalize,
                            float *logits, int32_t *ids, float *wts, hipStream_t st);
hipError_t launch_moe_plan(const int32_t *ids, int P, int E, int k, int tile_rows, int max_tiles, int32_t *offsets,
                           int32_t *sorted_tok, int32_t *pos_of, int32_t *tiles, int32_t *n_tiles, hipStream_t st);
hipError_t launch_moe_combine(const float *y, const int32_t *pos_of, const float *wts, const uint16_t *res,
                              uint16_t *out, int T, int d, int k, hipStream_t st);

}  // namespace eb
