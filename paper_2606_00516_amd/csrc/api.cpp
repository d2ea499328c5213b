// C ABI of libeb.so: handle, workspace carve-up, validation and the launch
// sequence of one decoder-layer step on the caller's stream.
#include <cmath>
#include <hip/hip_runtime.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include <string>
#include <vector>

#include "../../include/eb_layer.h"
#include "eb_internal.h"
#include "host_plan.h"

static_assert(eb::kDecInfo == eb::kDecInfoInts, "decode record layout");
static_assert(eb::kCombInfo == eb::kCombInfoInts, "combine record layout");

using namespace eb;

namespace {

thread_local std::string g_err;

eb_status fail(eb_status s, const std::string &msg) {
  g_err = msg;
  return s;
}

constexpr int kRing = 4;  // pinned staging slots per handle

// Stages of a step, in launch order (names returned by eb_profile_stage_name).
constexpr int kStages = 9;
const char *const kStageNames[kStages] = {"rmsnorm_1", "qkv_gemm", "rope_kv_append", "attention", "attention_combine",
                                          "o_gemm", "rmsnorm_2", "gate_up_gemm", "down_gemm"};

size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

Shape shape_of(const eb_layer_config &c) {
  Shape s{c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn, c.rms_eps, c.rope_theta};
  if (c.n_experts > 0) {
    s.ne = c.n_experts;
    s.topk = c.top_k;
    s.effn = c.expert_ffn;
    s.renorm = c.moe_renormalize ? 1 : 0;
  }
  s.qkn = c.qk_norm ? 1 : 0;
  return s;
}

namespace {
// Workspace of the MoE block: routing, the sorted order and tiles, the
// experts' SwiGLU outputs (bf16) and down products (fp32), 256-byte aligned.
struct MoeLayout {
  size_t logits, ids, wts, offsets, sorted_tok, pos_of, tiles, n_tiles, m, y, total;
  int max_tiles;
};
MoeLayout moe_layout(int T, int d, int E, int k, int F) {
  MoeLayout L{};
  const size_t P = (size_t)T * k;
  L.max_tiles = (int)((P + 63) / 64) + E;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.logits = take((size_t)T * E * 4);
  L.ids = take(P * 4);
  L.wts = take(P * 4);
  L.offsets = take((size_t)(E + 1) * 4);
  L.sorted_tok = take(P * 4);
  L.pos_of = take(P * 4);
  L.tiles = take((size_t)3 * L.max_tiles * 4);
  L.n_tiles = take(4);
  L.m = take(P * F * 2);
  L.y = take(P * d * 4);
  L.total = off;
  return L;
}
eb_status moe_limits(int T, int d, int E, int k, int F) {
  const size_t P = (size_t)T * k;
  (void)E;
  if ((size_t)T * d * 2 >= ((size_t)1 << 31) || P * F * 2 >= ((size_t)1 << 31) ||
      (size_t)2 * F * d * 2 >= ((size_t)1 << 31) || P >= ((size_t)1 << 30))
    return fail(EB_ERR_LIMITS, "MoE operands exceed the kernels' 32-bit ranges");
  return EB_OK;
}
eb_status check_moe(int T, int d, int E, int k, int F) {
  if (T < 0 || d <= 0 || E <= 0 || k <= 0 || F <= 0) return fail(EB_ERR_CONFIG, "MoE sizes must be positive");
  if (d % 32) return fail(EB_ERR_CONFIG, "MoE hidden size must be a multiple of 32");
  if (F % 8) return fail(EB_ERR_CONFIG, "MoE expert width must be a multiple of 8");
  if (E % 16 || E > 256) return fail(EB_ERR_CONFIG, "MoE expert count must be a multiple of 16, at most 256");
  if (k > E || k > 64) return fail(EB_ERR_CONFIG, "MoE top_k must be at most the expert count and 64");
  return moe_limits(T, d, E, k, F);
}

// The block on the stream: routing, the sorted order and the gate/up
// products (first), then the down products and the weighted combine with
// the residual (second); b is the block's input, out its output.
struct MoeArgs {
  const uint16_t *b, *res, *w_router, *w_gate_up, *w_down;
  uint16_t *out;
  int T, d, E, k, F, renorm;
  char *ws;
};
struct MoeBufs {
  float *logits, *wts, *y;
  int32_t *ids, *offsets, *sorted_tok, *pos_of, *tiles, *n_tiles;
  uint16_t *m;
  int max_tiles;
  bool big;
};
MoeBufs moe_bufs(const MoeArgs &a) {
  const MoeLayout L = moe_layout(a.T, a.d, a.E, a.k, a.F);
  MoeBufs B;
  B.logits = reinterpret_cast<float *>(a.ws + L.logits);
  B.ids = reinterpret_cast<int32_t *>(a.ws + L.ids);
  B.wts = reinterpret_cast<float *>(a.ws + L.wts);
  B.offsets = reinterpret_cast<int32_t *>(a.ws + L.offsets);
  B.sorted_tok = reinterpret_cast<int32_t *>(a.ws + L.sorted_tok);
  B.pos_of = reinterpret_cast<int32_t *>(a.ws + L.pos_of);
  B.tiles = reinterpret_cast<int32_t *>(a.ws + L.tiles);
  B.n_tiles = reinterpret_cast<int32_t *>(a.ws + L.n_tiles);
  B.m = reinterpret_cast<uint16_t *>(a.ws + L.m);
  B.y = reinterpret_cast<float *>(a.ws + L.y);
  B.max_tiles = L.max_tiles;
  // experts with a few rows each (decode batches) stream their weights in
  // 64-row tiles; with 128 or more rows per expert on average the 256 x 256
  // kernel takes tiles of up to 256 rows
  B.big = (long)a.T * a.k >= 128L * a.E && a.d % 64 == 0 && a.F % 64 == 0;
  return B;
}
hipError_t moe_first(const MoeArgs &a, hipStream_t st) {
  const MoeBufs B = moe_bufs(a);
  auto grouped = B.big ? launch_gemm_grouped_big : launch_gemm_grouped;
  hipError_t e = launch_moe_route(a.b, a.w_router, a.T, a.d, a.E, a.k, a.renorm, B.logits, B.ids, B.wts, st);
  if (e == hipSuccess)
    e = launch_moe_plan(B.ids, a.T * a.k, a.E, a.k, B.big ? 256 : 64, B.max_tiles, B.offsets, B.sorted_tok, B.pos_of,
                        B.tiles, B.n_tiles, st);
  if (e == hipSuccess)
    e = grouped(a.b, a.T, B.sorted_tok, a.w_gate_up, B.m, false, B.tiles, B.n_tiles, B.max_tiles, 2 * a.F, a.d,
                EPI_SILU_MUL, st);
  return e;
}
hipError_t moe_second(const MoeArgs &a, hipStream_t st) {
  const MoeBufs B = moe_bufs(a);
  auto grouped = B.big ? launch_gemm_grouped_big : launch_gemm_grouped;
  hipError_t e = grouped(B.m, a.T * a.k, nullptr, a.w_down, B.y, true, B.tiles, B.n_tiles, B.max_tiles, a.d, a.F,
                         EPI_STORE, st);
  if (e == hipSuccess) e = launch_moe_combine(B.y, B.pos_of, B.wts, a.res, a.out, a.T, a.d, a.k, st);
  return e;
}
}  // namespace

// Byte offsets of everything a step keeps in the caller's workspace.
struct WsLayout {
  size_t meta = 0, act = 0, qkv = 0, attn = 0, h1 = 0, mlp = 0, part_o = 0, part_ml = 0, gemm = 0, alt = 0,
         moe = 0, ssq = 0, total = 0;
};

// A decode-sized QKV projection (weight streaming with split K) takes the
// first RMSNorm into its operand staging and its split-K sum into the RoPE /
// append kernel: two launches fewer per layer.
bool fused_qkv(const GemmPlan &qp) { return qp.kind == 0 && qp.splits >= 2; }

// full_step: buffers of a whole layer; stack: plus the second activation
// buffer that consecutive layers of a stack alternate with y.
WsLayout layout_for(const Shape &s, const HostPlan &p, bool full_step, bool stack = false) {
  WsLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t T = (size_t)p.T;
  L.meta = take(p.blob.size() * sizeof(int32_t));
  L.part_o = take((size_t)p.total_splits * s.nkv * s.group() * s.hd * sizeof(float));
  L.part_ml = take((size_t)p.total_splits * s.nkv * s.group() * 2 * sizeof(float));
  if (full_step) {
    L.act = take(T * s.hidden * 2);
    L.qkv = take(T * s.qkv_cols() * 2);
    L.attn = take(T * s.nq * s.hd * 2);
    L.h1 = take(T * s.hidden * 2);
    if (!s.moe()) L.mlp = take(T * s.ffn * 2);
    size_t g = 0;
    const int M = p.T;
    // room for the plans of either weight type (the feed-forward ones when dense)
    for (int w8 = 0; w8 < 2; ++w8) {
      const int nplans = s.moe() ? 2 : 4;  // (an MoE layer has no dense feed-forward GEMMs)
      for (int i = 0; i < nplans; ++i) {
        const GemmPlan gp = i == 0   ? plan_gemm(M, s.qkv_cols(), s.hidden, EPI_STORE, w8)
                            : i == 1 ? plan_gemm(M, s.hidden, s.nq * s.hd, EPI_RESIDUAL, w8)
                            : i == 2 ? plan_gemm(M, 2 * s.ffn, s.hidden, EPI_SILU_MUL, w8)
                                     : plan_gemm(M, s.hidden, s.ffn, EPI_RESIDUAL, w8);
        g = gp.ws_bytes > g ? gp.ws_bytes : g;
      }
    }
    if (s.moe()) L.moe = take(moe_layout(p.T, s.hidden, s.ne, s.topk, s.effn).total);
    L.gemm = take(g);
    // row sums of squares of the fused first RMSNorm (either weight type)
    int ss_splits = 1;
    for (int w8 = 0; w8 < 2; ++w8) {
      const GemmPlan qp = plan_gemm(M, s.qkv_cols(), s.hidden, EPI_STORE, w8);
      if (fused_qkv(qp) && qp.splits > ss_splits) ss_splits = qp.splits;
    }
    L.ssq = take((size_t)ss_splits * T * sizeof(float));
    if (stack) L.alt = take(T * s.hidden * 2);
  }
  L.total = off;
  return L;
}

DevMeta meta_at(const HostPlan &p, const int32_t *dev) {
  DevMeta m;
  m.seq_ctx = dev + p.o_ctx;
  m.seq_len = dev + p.o_len;
  m.seq_row = dev + p.o_row;
  m.row_seq = dev + p.o_row_seq;
  m.row_pos = dev + p.o_row_pos;
  m.dec_info = dev + p.o_dec_info;
  m.dec_part = dev + p.o_part;
  m.dec_short = dev + p.o_short;
  m.comb_list = dev + p.o_comb;
  m.tile_seq = dev + p.o_tseq;
  m.tile_qb = dev + p.o_tqb;
  m.gather_off = dev + p.o_goff;
  m.S = p.S;
  m.T = p.T;
  m.n_dec = p.n_dec;
  m.total_splits = p.total_splits;
  m.total_units = p.total_units;
  m.n_comb = p.n_comb;
  m.n_tiles = p.n_tiles;
  m.n_full_units = p.n_full_units;
  m.n_part = p.n_part;
  m.n_short = p.n_short;
  return m;
}

eb_status hip_fail(hipError_t e, const char *what) {
  return fail(EB_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace

struct eb_handle {
  eb_layer_config cfg;
  Shape shape;
  int32_t max_seqs, max_tokens;
  int device;
  size_t slot_cap;  // int32 elements per pinned slot
  int32_t *pinned[kRing];
  hipEvent_t ev[kRing];
  bool used[kRing];
  int next;
  // per-stage timing (eb_profile): step j of a profiled run records into
  // slot j % prof_slots, where events [2 (l kStages + s)] and the next one
  // bracket stage s of layer l
  bool prof;
  uint32_t prof_mask;  // stages recorded (bit s: stage s)
  int prof_slots;
  long prof_count;  // steps recorded since profiling was switched on
  std::vector<std::vector<hipEvent_t>> pslot;
  std::vector<int> slot_layers;
  int max_layers;  // most layers a step on this handle has run
  // debug validation: every step copies the device block tables back and
  // checks them on the host before it enqueues anything (EB_DEBUG_VALIDATE)
  bool debug_validate;
  // device address of this device's fixed scratch (eb_layer_step_mixed_noalloc);
  // null with the lookup's error kept when it failed
  void *scratch;
  hipError_t scratch_err;
};

namespace {

// Copy a plan's metadata into the workspace through the next pinned slot,
// asynchronously on the stream.
eb_status stage_meta(eb_handle *h, const HostPlan &p, void *ws, const WsLayout &L, hipStream_t st) {
  const int k = h->next;
  h->next = (h->next + 1) % kRing;
  if (p.blob.size() > h->slot_cap) return fail(EB_ERR_LIMITS, "step metadata exceeds the handle's staging buffer");
  if (h->used[k]) {
    hipError_t e = hipEventSynchronize(h->ev[k]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  }
  memcpy(h->pinned[k], p.blob.data(), p.blob.size() * sizeof(int32_t));
  hipError_t e = hipMemcpyAsync(static_cast<char *>(ws) + L.meta, h->pinned[k], p.blob.size() * sizeof(int32_t),
                                hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(metadata)");
  e = hipEventRecord(h->ev[k], st);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  h->used[k] = true;
  return EB_OK;
}

eb_status check_kv(const eb_kv_cache *kv) {
  if (!kv) return fail(EB_ERR_NULL, "kv is NULL");
  if (!kv->k_cache || !kv->v_cache || !kv->block_tables) return fail(EB_ERR_NULL, "kv cache or block table is NULL");
  if (kv->num_pages <= 0 || kv->max_pages_per_seq <= 0)
    return fail(EB_ERR_PAGES, "num_pages and max_pages_per_seq must be positive");
  if (kv->kv_dtype != EB_KV_BF16 && kv->kv_dtype != EB_KV_FP8_E4M3) return fail(EB_ERR_CONFIG, "unknown kv_dtype");
  if (kv->kv_dtype == EB_KV_FP8_E4M3 &&
      !(std::isfinite(kv->k_scale) && kv->k_scale > 0.f && std::isfinite(kv->v_scale) && kv->v_scale > 0.f))
    return fail(EB_ERR_CONFIG, "an 8-bit cache needs finite positive k_scale and v_scale");
  return EB_OK;
}

eb_status check_common(const eb_handle *h, const eb_batch *b, eb_mode mode, int32_t max_pages) {
  if (!h) return fail(EB_ERR_NULL, "handle is NULL");
  std::string err;
  eb_status s = check_batch(h->cfg, b, max_pages, mode, err);
  if (s != EB_OK) return fail(s, err);
  if (b->num_seqs > h->max_seqs || b->num_tokens > h->max_tokens)
    return fail(EB_ERR_LIMITS, "batch larger than the handle's max_seqs / max_tokens");
  return EB_OK;
}

eb_status check_ws(void *ws, size_t ws_bytes, size_t need) {
  if (need == 0) return EB_OK;
  if (!ws) return fail(EB_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(EB_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return fail(EB_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes, got " +
                                      std::to_string(ws_bytes));
  return EB_OK;
}

// Debug validation of device block tables (handles created with
// EB_DEBUG_VALIDATE set): copy the needed rows back on the caller's stream,
// wait for them and run the host check.  Release handles skip this: they
// never read device block tables on the host.
eb_status debug_check_tables(const eb_handle *h, const eb_batch *b, const eb_kv_cache *kv, int n, hipStream_t st) {
  if (!h->debug_validate || b->num_seqs == 0) return EB_OK;
  std::vector<int32_t> host;
  for (int l = 0; l < n; ++l) {
    const size_t cnt = (size_t)b->num_seqs * kv[l].max_pages_per_seq;
    host.resize(cnt);
    hipError_t e = hipMemcpyAsync(host.data(), kv[l].block_tables, cnt * sizeof(int32_t), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail(EB_ERR_HIP, std::string("debug validation copy: ") + hipGetErrorString(e));
    std::string err;
    const eb_status s = check_tables(h->cfg, *b, host.data(), kv[l].num_pages, kv[l].max_pages_per_seq, err);
    if (s != EB_OK) return fail(s, (n > 1 ? "layer " + std::to_string(l) + ": " : std::string()) + err);
  }
  return EB_OK;
}

KV kv_of(const eb_kv_cache *kv) {
  const bool f8 = kv->kv_dtype == EB_KV_FP8_E4M3;
  return KV{static_cast<uint16_t *>(kv->k_cache), static_cast<uint16_t *>(kv->v_cache), kv->block_tables,
            kv->num_pages, kv->max_pages_per_seq, f8 ? 1 : 0, f8 ? kv->k_scale : 1.f, f8 ? kv->v_scale : 1.f};
}

// The weights of one layer for a batch of T tokens: pointers, the weight
// type, and (8-bit weights) scales and that a kernel takes every projection.
eb_status check_weights(const eb_layer_weights *w, const Shape &sh, int T) {
  if (!w || !w->attn_norm || !w->w_qkv || !w->w_o || !w->mlp_norm)
    return fail(EB_ERR_NULL, "a weight pointer is NULL");
  if (sh.qkn && (!w->q_norm || !w->k_norm)) return fail(EB_ERR_NULL, "q_norm or k_norm is NULL");
  if (sh.moe()) {
    if (!w->w_router || !w->w_experts_gate_up || !w->w_experts_down)
      return fail(EB_ERR_NULL, "a mixture-of-experts weight pointer is NULL");
    if (w->w_dtype != EB_W_BF16) return fail(EB_ERR_CONFIG, "mixture-of-experts layers take bf16 weights");
    if (moe_limits(T, sh.hidden, sh.ne, sh.topk, sh.effn) != EB_OK) return EB_ERR_LIMITS;
    return EB_OK;
  }
  if (!w->w_gate_up || !w->w_down) return fail(EB_ERR_NULL, "a weight pointer is NULL");
  if (w->w_dtype == EB_W_BF16) return EB_OK;
  if (w->w_dtype != EB_W_FP8_E4M3) return fail(EB_ERR_CONFIG, "unknown w_dtype");
  const float *sc[4] = {w->s_qkv, w->s_o, w->s_gate_up, w->s_down};
  for (const float *p : sc) {
    if (!p) return fail(EB_ERR_NULL, "8-bit weights need the four row-scale pointers");
    if (reinterpret_cast<uintptr_t>(p) % 16) return fail(EB_ERR_CONFIG, "row scales must be 16-byte aligned");
  }
  const int shp[4][3] = {{sh.qkv_cols(), sh.hidden, EPI_STORE},
                         {sh.hidden, sh.nq * sh.hd, EPI_RESIDUAL},
                         {2 * sh.ffn, sh.hidden, EPI_SILU_MUL},
                         {sh.hidden, sh.ffn, EPI_RESIDUAL}};
  for (const auto &g : shp)
    if (plan_gemm(T, g[0], g[1], g[2], true).kind < 0)
      return fail(EB_ERR_LIMITS, "8-bit projection too large for the GEMM kernels");
  return EB_OK;
}

// Workspace buffers of one layer body.
struct StepBufs {
  uint16_t *act, *qkv, *attn, *h1, *mlp, *alt;
  float *part_o, *part_ml;
  void *gws;
  char *moe;
  float *ssq;
};

StepBufs bufs_at(char *base, const WsLayout &L) {
  return StepBufs{reinterpret_cast<uint16_t *>(base + L.act),  reinterpret_cast<uint16_t *>(base + L.qkv),
                  reinterpret_cast<uint16_t *>(base + L.attn), reinterpret_cast<uint16_t *>(base + L.h1),
                  reinterpret_cast<uint16_t *>(base + L.mlp),  L.alt ? reinterpret_cast<uint16_t *>(base + L.alt)
                                                                      : nullptr,
                  reinterpret_cast<float *>(base + L.part_o), reinterpret_cast<float *>(base + L.part_ml),
                  base + L.gemm, base + L.moe, reinterpret_cast<float *>(base + L.ssq)};
}

// Make sure a profiling slot's events cover n layers.  They only time the
// stages: recording them skips the system-scope fence (an L2 write-back and
// invalidation that would perturb the very work being timed).
eb_status grow_events(std::vector<hipEvent_t> &pev, int layers) {
  const size_t need = (size_t)2 * kStages * layers;
  while (pev.size() < need) {
    hipEvent_t e = nullptr;
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) return hip_fail(r, "hipEventCreate");
    pev.push_back(e);
  }
  return EB_OK;
}

// The nine stages of one layer on the stream: x -> y with weights w and
// cache kvd; the batch metadata m is already in the workspace.
static inline const uint16_t *pk(const void *p) { return static_cast<const uint16_t *>(p); }

eb_status layer_body(eb_handle *h, const eb_layer_weights *w, const KV &kvd, const DevMeta &m, const StepBufs &B,
                     const uint16_t *xin, uint16_t *yout, int T, eb_mode mode, int layer, hipEvent_t *pev,
                     hipStream_t st) {
  const Shape &sh = h->shape;
  const bool w8 = w->w_dtype == EB_W_FP8_E4M3;
  hipError_t e;
  auto mark = [&](int i) -> hipError_t {
    return pev && ((h->prof_mask >> (i / 2)) & 1u) ? hipEventRecord(pev[(size_t)2 * kStages * layer + i], st)
                                                   : hipSuccess;
  };
#define EB_STAGE(idx, call, what)                                       \
  if ((e = mark(2 * (idx))) != hipSuccess) return hip_fail(e, "hipEventRecord"); \
  if ((e = (call)) != hipSuccess) return hip_fail(e, what);              \
  if ((e = mark(2 * (idx) + 1)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  const GemmPlan qp = plan_gemm(T, sh.qkv_cols(), sh.hidden, EPI_STORE, w8);
  const uint16_t *g1 = static_cast<const uint16_t *>(w->attn_norm);
  const uint16_t *gq = static_cast<const uint16_t *>(w->q_norm), *gk = static_cast<const uint16_t *>(w->k_norm);
  if (fused_qkv(qp)) {
    // the first RMSNorm rides in the projection, the split-K sum in the RoPE
    // kernel (stage 0 stays empty)
    EB_STAGE(0, hipSuccess, "rmsnorm1");
    EB_STAGE(1,
             launch_gemm_prenorm(qp, xin, g1, w->w_qkv, w8 ? w->s_qkv : nullptr, T, sh.qkv_cols(), sh.hidden,
                                 static_cast<float *>(B.gws), B.ssq, st, w8 ? nullptr : pk(w->p_qkv)),
             "qkv gemm");
    EB_STAGE(2, launch_qkv_rope_append(sh, static_cast<const float *>(B.gws), qp.splits, B.ssq, B.qkv, kvd, m, st, gq, gk),
             "rope/kv append");
  } else {
    EB_STAGE(0, launch_rmsnorm(xin, g1, B.act, T, sh.hidden, sh.eps, st), "rmsnorm1");
    EB_STAGE(1,
             launch_gemm(qp, B.act, w->w_qkv, w8 ? w->s_qkv : nullptr, B.qkv, nullptr, T, sh.qkv_cols(), sh.hidden,
                         EPI_STORE, B.gws, st, nullptr, w8 ? nullptr : pk(w->p_qkv)),
             "qkv gemm");
    EB_STAGE(2, launch_rope_append(sh, B.qkv, kvd, m, st, gq, gk), "rope/kv append");
  }
  const int kind = mode == EB_MODE_DECODE ? 0 : (mode == EB_MODE_PREFILL ? 1 : 2);
  EB_STAGE(3, launch_attention(sh, B.qkv, kvd, m, B.attn, B.part_o, B.part_ml, kind, st, 1), "attention");
  EB_STAGE(4, launch_attention(sh, B.qkv, kvd, m, B.attn, B.part_o, B.part_ml, kind, st, 2), "attention combine");
  // when the O projection splits K (decode-sized batches) its split-K sum
  // also writes RMSNorm(h1) * g2, and stage 6 has nothing left to do
  NormFuse nf{static_cast<const uint16_t *>(w->mlp_norm), B.act, sh.eps, false};
  EB_STAGE(5,
           launch_gemm(plan_gemm(T, sh.hidden, sh.nq * sh.hd, EPI_RESIDUAL, w8), B.attn, w->w_o,
                       w8 ? w->s_o : nullptr, B.h1, xin, T, sh.hidden, sh.nq * sh.hd, EPI_RESIDUAL, B.gws, st, &nf,
                       w8 ? nullptr : pk(w->p_o)),
           "o gemm");
  EB_STAGE(6,
           nf.done ? hipSuccess
                   : launch_rmsnorm(B.h1, static_cast<const uint16_t *>(w->mlp_norm), B.act, T, sh.hidden, sh.eps, st),
           "rmsnorm2");
  if (sh.moe()) {
    // the mixture-of-experts block: stage 7 routes and runs the gate/up
    // products, stage 8 the down products and the combine with h1
    const MoeArgs ma{B.act, B.h1, static_cast<const uint16_t *>(w->w_router),
                     static_cast<const uint16_t *>(w->w_experts_gate_up),
                     static_cast<const uint16_t *>(w->w_experts_down), yout, T, sh.hidden, sh.ne, sh.topk, sh.effn,
                     sh.renorm, B.moe};
    EB_STAGE(7, moe_first(ma, st), "moe routing and gate/up");
    EB_STAGE(8, moe_second(ma, st), "moe down and combine");
    return EB_OK;
  }
  EB_STAGE(7,
           launch_gemm(plan_gemm(T, 2 * sh.ffn, sh.hidden, EPI_SILU_MUL, w8), B.act, w->w_gate_up,
                       w8 ? w->s_gate_up : nullptr, B.mlp, nullptr, T, 2 * sh.ffn, sh.hidden, EPI_SILU_MUL, B.gws,
                       st, nullptr, w8 ? nullptr : pk(w->p_gate_up)),
           "gate/up gemm");
  EB_STAGE(8,
           launch_gemm(plan_gemm(T, sh.hidden, sh.ffn, EPI_RESIDUAL, w8), B.mlp, w->w_down,
                       w8 ? w->s_down : nullptr, yout, B.h1, T, sh.hidden, sh.ffn, EPI_RESIDUAL, B.gws, st, nullptr,
                       w8 ? nullptr : pk(w->p_down)),
           "down gemm");
#undef EB_STAGE
  return EB_OK;
}

// n_layers layer bodies over one planned batch: layer l reads x (l = 0) or
// the previous layer's output and writes y or the alternate buffer, so that
// the last layer writes y.  Every check runs before anything is enqueued.
eb_status run_layers(eb_handle *h, int32_t n_layers, const eb_layer_weights *w, const eb_kv_cache *kv,
                     const eb_batch *b, const void *x, void *y, void *ws, size_t ws_bytes, void *stream,
                     eb_mode mode, bool allow_prof = true) {
  if (!h) return fail(EB_ERR_NULL, "handle is NULL");
  if (n_layers < 1) return fail(EB_ERR_CONFIG, "n_layers must be >= 1");
  if (!w || !kv) return fail(EB_ERR_NULL, "weights or kv is NULL");
  int32_t min_pages = 0;
  const int T = b && b->num_tokens > 0 ? b->num_tokens : 1;  // (b itself is checked below)
  for (int l = 0; l < n_layers; ++l) {
    eb_status s = check_weights(&w[l], h->shape, T);
    if (s == EB_OK) s = check_kv(&kv[l]);
    if (s != EB_OK) return n_layers > 1 ? fail(s, "layer " + std::to_string(l) + ": " + g_err) : s;
    min_pages = l == 0 ? kv[l].max_pages_per_seq : std::min(min_pages, kv[l].max_pages_per_seq);
  }
  eb_status s = check_common(h, b, mode, min_pages);
  if (s != EB_OK) return s;
  if (b->num_tokens == 0) return EB_OK;
  if (n_layers > h->max_layers) h->max_layers = n_layers;
  if (!x || !y) return fail(EB_ERR_NULL, "x or y is NULL");
  if (x == y) return fail(EB_ERR_BATCH, "y must not alias x");
  s = debug_check_tables(h, b, kv, n_layers, static_cast<hipStream_t>(stream));
  if (s != EB_OK) return s;
  HostPlan p;
  build_plan(h->cfg, *b, mode, p);
  const bool stack = n_layers > 1;
  const WsLayout L = layout_for(h->shape, p, true, stack);
  s = check_ws(ws, ws_bytes, L.total);
  if (s != EB_OK) return s;
  const int slot = h->prof && allow_prof ? (int)(h->prof_count % h->prof_slots) : -1;
  if (slot >= 0) {
    s = grow_events(h->pslot[slot], n_layers);
    if (s != EB_OK) return s;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  char *base = static_cast<char *>(ws);
  s = stage_meta(h, p, ws, L, st);
  if (s != EB_OK) return s;
  const DevMeta m = meta_at(p, reinterpret_cast<const int32_t *>(base + L.meta));
  const StepBufs B = bufs_at(base, L);
  const uint16_t *in = static_cast<const uint16_t *>(x);
  for (int l = 0; l < n_layers; ++l) {
    uint16_t *out = ((n_layers - 1 - l) % 2 == 0) ? static_cast<uint16_t *>(y) : B.alt;
    s = layer_body(h, &w[l], kv_of(&kv[l]), m, B, in, out, p.T, mode, l,
                   slot >= 0 ? h->pslot[slot].data() : nullptr, st);
    if (s != EB_OK) return s;
    in = out;
  }
  if (slot >= 0) {
    h->slot_layers[slot] = n_layers;
    ++h->prof_count;
  }
  return EB_OK;
}

}  // namespace

extern "C" {

const char *eb_status_str(eb_status s) {
  switch (s) {
    case EB_OK: return "EB_OK";
    case EB_ERR_NULL: return "EB_ERR_NULL";
    case EB_ERR_CONFIG: return "EB_ERR_CONFIG";
    case EB_ERR_BATCH: return "EB_ERR_BATCH";
    case EB_ERR_MODE: return "EB_ERR_MODE";
    case EB_ERR_PAGES: return "EB_ERR_PAGES";
    case EB_ERR_WORKSPACE: return "EB_ERR_WORKSPACE";
    case EB_ERR_LIMITS: return "EB_ERR_LIMITS";
    case EB_ERR_HIP: return "EB_ERR_HIP";
  }
  return "unknown status";
}

const char *eb_last_error(void) { return g_err.c_str(); }

eb_status eb_create(const eb_layer_config *cfg, int32_t max_seqs, int32_t max_tokens, eb_handle **out) {
  if (!out) return fail(EB_ERR_NULL, "out is NULL");
  *out = nullptr;
  std::string err;
  eb_status s = check_config(cfg, err);
  if (s != EB_OK) return fail(s, err);
  if (max_seqs < 1 || max_tokens < 1) return fail(EB_ERR_LIMITS, "max_seqs and max_tokens must be >= 1");
  eb_handle *h = new eb_handle();
  h->cfg = *cfg;
  h->shape = shape_of(*cfg);
  h->max_seqs = max_seqs;
  h->max_tokens = max_tokens;
  h->next = 0;
  hipError_t e = hipGetDevice(&h->device);
  if (e != hipSuccess) {
    delete h;
    return hip_fail(e, "hipGetDevice");
  }
  h->slot_cap = plan_capacity(max_seqs, max_tokens, cfg->n_q_heads / cfg->n_kv_heads);
  h->prof = false;
  h->prof_slots = 0;
  h->prof_mask = 0;
  h->prof_count = 0;
  h->max_layers = 1;
#ifdef EB_DEBUG_VALIDATE
  h->debug_validate = true;
#else
  const char *dv = getenv("EB_DEBUG_VALIDATE");
  h->debug_validate = dv && dv[0] && strcmp(dv, "0") != 0;
#endif
  for (int k = 0; k < kRing; ++k) {
    h->pinned[k] = nullptr;
    h->ev[k] = nullptr;
    h->used[k] = false;
  }
  h->scratch_err = noalloc_scratch_setup(h->device, &h->scratch);
  for (int k = 0; k < kRing; ++k) {
    e = hipHostMalloc(reinterpret_cast<void **>(&h->pinned[k]), h->slot_cap * sizeof(int32_t), hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->ev[k], hipEventDisableTiming);
    if (e != hipSuccess) {
      eb_destroy(h);
      return hip_fail(e, "pinned staging allocation");
    }
  }
  *out = h;
  return EB_OK;
}

void eb_destroy(eb_handle *h) {
  if (!h) return;
  for (int k = 0; k < kRing; ++k) {
    if (h->ev[k]) {
      if (h->used[k]) (void)hipEventSynchronize(h->ev[k]);
      (void)hipEventDestroy(h->ev[k]);
    }
    if (h->pinned[k]) (void)hipHostFree(h->pinned[k]);
  }
  for (auto &pev : h->pslot)
    for (hipEvent_t e : pev) (void)hipEventDestroy(e);
  delete h;
}

size_t eb_workspace_bytes(const eb_handle *h, const eb_batch *batch, eb_mode mode) {
  if (!h) return 0;
  std::string err;
  if (check_batch(h->cfg, batch, -1, mode, err) != EB_OK) return 0;
  HostPlan p;
  build_plan(h->cfg, *batch, mode, p);
  return layout_for(h->shape, p, true).total;
}

size_t eb_workspace_offset(const eb_handle *h, const eb_batch *batch, eb_mode mode, int32_t which) {
  const size_t none = (size_t)-1;
  if (!h) return none;
  std::string err;
  if (check_batch(h->cfg, batch, -1, mode, err) != EB_OK || batch->num_tokens == 0) return none;
  HostPlan p;
  build_plan(h->cfg, *batch, mode, p);
  const WsLayout L = layout_for(h->shape, p, true);
  switch (which) {
    case EB_WS_QKV: return L.qkv;
    case EB_WS_ATTN: return L.attn;
    case EB_WS_H1: return L.h1;
    case EB_WS_MLP: return h->shape.moe() ? none : L.mlp;
    case EB_WS_NORM: return L.act;
  }
  return none;
}

eb_status eb_layer_step_decode(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv, const eb_batch *batch,
                               const void *x, void *y, void *ws, size_t ws_bytes, void *stream) {
  return run_layers(h, 1, w, kv, batch, x, y, ws, ws_bytes, stream, EB_MODE_DECODE);
}

eb_status eb_layer_step_prefill(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv, const eb_batch *batch,
                                const void *x, void *y, void *ws, size_t ws_bytes, void *stream) {
  return run_layers(h, 1, w, kv, batch, x, y, ws, ws_bytes, stream, EB_MODE_PREFILL);
}

eb_status eb_layer_step_mixed(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv, const eb_batch *batch,
                              const void *x, void *y, void *ws, size_t ws_bytes, void *stream) {
  return run_layers(h, 1, w, kv, batch, x, y, ws, ws_bytes, stream, EB_MODE_MIXED);
}

size_t eb_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

eb_status eb_layer_step_mixed_noalloc(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv,
                                      const eb_batch *batch, const void *x, void *y, void *stream) {
  if (!h) return fail(EB_ERR_NULL, "handle is NULL");
  std::string err;
  eb_status s = check_batch(h->cfg, batch, -1, EB_MODE_MIXED, err);
  if (s != EB_OK) return fail(s, err);
  if (batch->num_tokens > 0) {
    HostPlan p;
    build_plan(h->cfg, *batch, EB_MODE_MIXED, p);
    const size_t need = layout_for(h->shape, p, true).total;
    if (need > kNoAllocScratchBytes)
      return fail(EB_ERR_WORKSPACE, "batch needs " + std::to_string(need) + " bytes of workspace, the fixed scratch holds " +
                                        std::to_string(kNoAllocScratchBytes));
  }
  if (!h->scratch) return hip_fail(h->scratch_err, "fixed scratch address (hipGetSymbolAddress)");
  return run_layers(h, 1, w, kv, batch, x, y, h->scratch, kNoAllocScratchBytes, stream, EB_MODE_MIXED, false);
}

size_t eb_stack_workspace_bytes(const eb_handle *h, const eb_batch *batch, eb_mode mode) {
  if (!h) return 0;
  std::string err;
  if (check_batch(h->cfg, batch, -1, mode, err) != EB_OK) return 0;
  HostPlan p;
  build_plan(h->cfg, *batch, mode, p);
  return layout_for(h->shape, p, true, true).total;
}

eb_status eb_stack_step(eb_handle *h, eb_mode mode, int32_t n_layers, const eb_layer_weights *weights,
                        const eb_kv_cache *kv, const eb_batch *batch, const void *x, void *y, void *ws,
                        size_t ws_bytes, void *stream) {
  if (mode != EB_MODE_DECODE && mode != EB_MODE_PREFILL && mode != EB_MODE_MIXED)
    return fail(EB_ERR_MODE, "unknown mode");
  return run_layers(h, n_layers, weights, kv, batch, x, y, ws, ws_bytes, stream, mode);
}

eb_status eb_validate(const eb_layer_config *cfg, const eb_batch *batch, const int32_t *block_tables_host,
                      int32_t num_pages, int32_t max_pages_per_seq, eb_mode mode) {
  std::string err;
  eb_status s = check_config(cfg, err);
  if (s != EB_OK) return fail(s, err);
  if (max_pages_per_seq <= 0 || num_pages <= 0)
    return fail(EB_ERR_PAGES, "num_pages and max_pages_per_seq must be positive");
  s = check_batch(*cfg, batch, max_pages_per_seq, mode, err);
  if (s != EB_OK) return fail(s, err);
  s = check_tables(*cfg, *batch, block_tables_host, num_pages, max_pages_per_seq, err);
  if (s != EB_OK) return fail(s, err);
  return EB_OK;
}

eb_status eb_profile(eb_handle *h, int32_t steps, uint32_t stage_mask) {
  if (!h) return fail(EB_ERR_NULL, "handle is NULL");
  if (steps < 0) return fail(EB_ERR_CONFIG, "steps must be >= 0");
  const uint32_t all = (1u << kStages) - 1u;
  if (stage_mask & ~all) return fail(EB_ERR_CONFIG, "stage_mask names an unknown stage");
  if (steps > 0) {
    // every slot's events exist before the first profiled step, for as many
    // layers as the handle's largest step so far (a larger step adds its own)
    if ((int)h->pslot.size() < steps) h->pslot.resize(steps);
    for (int k = 0; k < steps; ++k) {
      eb_status s = grow_events(h->pslot[k], h->max_layers);
      if (s != EB_OK) return s;
    }
    h->slot_layers.assign(steps, 0);
  }
  h->prof = steps > 0;
  h->prof_mask = stage_mask ? stage_mask : all;
  h->prof_slots = steps;
  h->prof_count = 0;
  return EB_OK;
}

int32_t eb_profile_read(eb_handle *h, float *ms, int32_t cap) {
  if (!h || !h->prof || h->prof_count == 0) return 0;
  const int nrec = h->prof_count < h->prof_slots ? (int)h->prof_count : h->prof_slots;
  int last_stage = kStages - 1;
  while (!((h->prof_mask >> last_stage) & 1u)) --last_stage;
  for (int k = 0; k < nrec; ++k) {
    const size_t last = (size_t)2 * (kStages * (h->slot_layers[k] - 1) + last_stage) + 1;
    if (hipEventSynchronize(h->pslot[k][last]) != hipSuccess) return -1;
  }
  const int n = cap < kStages ? cap : kStages;
  for (int i = 0; i < n; ++i) {
    double sum = 0.0;
    if (!((h->prof_mask >> i) & 1u)) {
      ms[i] = 0.f;
      continue;
    }
    for (int k = 0; k < nrec; ++k)
      for (int l = 0; l < h->slot_layers[k]; ++l) {
        const size_t b = (size_t)2 * (l * kStages + i);
        float t = 0.f;
        if (hipEventElapsedTime(&t, h->pslot[k][b], h->pslot[k][b + 1]) != hipSuccess) return -1;
        sum += t;
      }
    ms[i] = (float)(sum / nrec);
  }
  return n;
}

const char *eb_profile_stage_name(int32_t i) { return (i >= 0 && i < kStages) ? kStageNames[i] : nullptr; }

// ---------------------------------------------------------------------------
// single operations
// ---------------------------------------------------------------------------
eb_status eb_op_rmsnorm(const eb_handle *h, const void *x, const void *gamma, void *out, int32_t rows, void *stream) {
  if (!h) return fail(EB_ERR_NULL, "handle is NULL");
  if (rows < 0) return fail(EB_ERR_BATCH, "rows must be >= 0");
  if (rows == 0) return EB_OK;
  if (!x || !gamma || !out) return fail(EB_ERR_NULL, "x, gamma or out is NULL");
  hipError_t e = launch_rmsnorm(static_cast<const uint16_t *>(x), static_cast<const uint16_t *>(gamma),
                                static_cast<uint16_t *>(out), rows, h->shape.hidden, h->shape.eps,
                                static_cast<hipStream_t>(stream));
  return e == hipSuccess ? EB_OK : hip_fail(e, "rmsnorm");
}

size_t eb_op_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  size_t g = 0;
  for (int w8 = 0; w8 < 2; ++w8)
    for (int epi = 0; epi < 3; ++epi) {
      const size_t b = plan_gemm(M, N, K, epi, w8).ws_bytes;
      g = b > g ? b : g;
    }
  return g;
}

namespace {
eb_status op_gemm(const void *A, const void *W, const float *wscale, void *out, const void *residual, int32_t M,
                  int32_t N, int32_t K, eb_epilogue epi, void *ws, size_t ws_bytes, void *stream) {
  if (M < 0 || N <= 0 || K <= 0) return fail(EB_ERR_CONFIG, "M must be >= 0, N and K > 0");
  if (K % 8 || N % 8) return fail(EB_ERR_CONFIG, "N and K must be multiples of 8");
  if (epi != EB_EPI_STORE && epi != EB_EPI_RESIDUAL && epi != EB_EPI_SILU_MUL)
    return fail(EB_ERR_CONFIG, "unknown epilogue");
  if (epi == EB_EPI_SILU_MUL && N % 2) return fail(EB_ERR_CONFIG, "SiLU epilogue needs an even N");
  if (M == 0) return EB_OK;
  if (!A || !W || !out) return fail(EB_ERR_NULL, "A, W or out is NULL");
  if (epi == EB_EPI_RESIDUAL && !residual) return fail(EB_ERR_NULL, "residual is NULL");
  const bool w8 = wscale != nullptr;
  if (w8 && reinterpret_cast<uintptr_t>(wscale) % 16) return fail(EB_ERR_CONFIG, "row scales must be 16-byte aligned");
  const GemmPlan p = plan_gemm(M, N, K, (int)epi, w8);
  if (p.kind < 0) return fail(EB_ERR_LIMITS, "operands too large for the 8-bit GEMM kernels");
  eb_status s = check_ws(ws, ws_bytes, p.ws_bytes);
  if (s != EB_OK) return s;
  hipError_t e = launch_gemm(p, static_cast<const uint16_t *>(A), W, wscale, static_cast<uint16_t *>(out),
                             static_cast<const uint16_t *>(residual), M, N, K, (int)epi, ws,
                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? EB_OK : hip_fail(e, "gemm");
}
}  // namespace

eb_status eb_op_gemm(const void *A, const void *W, void *out, const void *residual, int32_t M, int32_t N, int32_t K,
                     eb_epilogue epi, void *ws, size_t ws_bytes, void *stream) {
  return op_gemm(A, W, nullptr, out, residual, M, N, K, epi, ws, ws_bytes, stream);
}

size_t eb_packed_weight_bytes(int rows, int cols) {
  if (rows <= 0 || cols <= 0 || rows % 16 || cols % 32) return 0;
  if ((size_t)rows * cols * 2 >= ((size_t)1 << 31)) return 0;
  return packed_weight_bytes(rows, cols);
}

eb_status eb_pack_weight(const void *w, void *packed, int rows, int cols, void *stream) {
  if (!w || !packed) return fail(EB_ERR_NULL, "w or packed is NULL");
  if (eb_packed_weight_bytes(rows, cols) == 0) return fail(EB_ERR_CONFIG, "shape has no packed form");
  const hipError_t e = pack_weight(static_cast<const uint16_t *>(w), static_cast<uint16_t *>(packed), rows, cols,
                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? EB_OK : fail(EB_ERR_HIP, hipGetErrorString(e));
}

eb_status eb_op_gemm_w8(const void *A, const void *W, const float *w_scale, void *out, const void *residual,
                        int32_t M, int32_t N, int32_t K, eb_epilogue epi, void *ws, size_t ws_bytes, void *stream) {
  if (!w_scale && M > 0) return fail(EB_ERR_NULL, "w_scale is NULL");
  return op_gemm(A, W, w_scale, out, residual, M, N, K, epi, ws, ws_bytes, stream);
}


size_t eb_op_moe_ffn_workspace_bytes(int32_t T, int32_t d, int32_t E, int32_t top_k, int32_t F) {
  if (T <= 0 || d <= 0 || E <= 0 || top_k <= 0 || F <= 0) return 0;
  return moe_layout(T, d, E, top_k, F).total;
}

eb_status eb_op_moe_ffn(const void *b, const void *residual, const void *w_router, const void *w_gate_up,
                        const void *w_down, int32_t T, int32_t d, int32_t E, int32_t top_k, int32_t F,
                        int32_t renormalize, void *out, int32_t *ids_out, float *weights_out, void *ws,
                        size_t ws_bytes, void *stream) {
  eb_status s = check_moe(T, d, E, top_k, F);
  if (s != EB_OK) return s;
  if (T == 0) return EB_OK;
  if (!b || !w_router || !w_gate_up || !w_down || !out) return fail(EB_ERR_NULL, "an input or out is NULL");
  s = check_ws(ws, ws_bytes, moe_layout(T, d, E, top_k, F).total);
  if (s != EB_OK) return s;
  const MoeArgs ma{static_cast<const uint16_t *>(b), static_cast<const uint16_t *>(residual),
                   static_cast<const uint16_t *>(w_router), static_cast<const uint16_t *>(w_gate_up),
                   static_cast<const uint16_t *>(w_down), static_cast<uint16_t *>(out), T, d, E, top_k, F,
                   renormalize ? 1 : 0, static_cast<char *>(ws)};
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const MoeBufs B = moe_bufs(ma);
  const size_t P = (size_t)T * top_k;
  hipError_t e = moe_first(ma, st);
  if (e == hipSuccess) e = moe_second(ma, st);
  if (e == hipSuccess && ids_out) e = hipMemcpyAsync(ids_out, B.ids, P * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess && weights_out) e = hipMemcpyAsync(weights_out, B.wts, P * 4, hipMemcpyDeviceToDevice, st);
  return e == hipSuccess ? EB_OK : hip_fail(e, "moe ffn");
}

eb_status eb_op_rope_kv_append(eb_handle *h, void *qkv, const eb_kv_cache *kv, const eb_batch *batch, void *ws,
                               size_t ws_bytes, void *stream) {
  eb_status s = check_kv(kv);
  if (s != EB_OK) return s;
  s = check_common(h, batch, EB_MODE_MIXED, kv->max_pages_per_seq);
  if (s != EB_OK) return s;
  if (batch->num_tokens == 0) return EB_OK;
  if (!qkv) return fail(EB_ERR_NULL, "qkv is NULL");
  if (h->shape.qkn) return fail(EB_ERR_CONFIG, "qk_norm layers: the norm gains come with the layer step entry points");
  s = debug_check_tables(h, batch, kv, 1, static_cast<hipStream_t>(stream));
  if (s != EB_OK) return s;
  HostPlan p;
  build_plan(h->cfg, *batch, EB_MODE_MIXED, p);
  const WsLayout L = layout_for(h->shape, p, false);
  s = check_ws(ws, ws_bytes, L.total);
  if (s != EB_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = stage_meta(h, p, ws, L, st);
  if (s != EB_OK) return s;
  const DevMeta m = meta_at(p, reinterpret_cast<const int32_t *>(static_cast<char *>(ws) + L.meta));
  hipError_t e = launch_rope_append(h->shape, static_cast<uint16_t *>(qkv), kv_of(kv), m, st);
  return e == hipSuccess ? EB_OK : hip_fail(e, "rope/kv append");
}

eb_status eb_op_attention(eb_handle *h, const void *qkv, const eb_kv_cache *kv, const eb_batch *batch, void *out,
                          void *ws, size_t ws_bytes, eb_mode mode, void *stream) {
  eb_status s = check_kv(kv);
  if (s != EB_OK) return s;
  s = check_common(h, batch, mode, kv->max_pages_per_seq);
  if (s != EB_OK) return s;
  if (batch->num_tokens == 0) return EB_OK;
  if (!qkv || !out) return fail(EB_ERR_NULL, "qkv or out is NULL");
  s = debug_check_tables(h, batch, kv, 1, static_cast<hipStream_t>(stream));
  if (s != EB_OK) return s;
  HostPlan p;
  build_plan(h->cfg, *batch, mode, p);
  const WsLayout L = layout_for(h->shape, p, false);
  s = check_ws(ws, ws_bytes, L.total);
  if (s != EB_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = stage_meta(h, p, ws, L, st);
  if (s != EB_OK) return s;
  char *base = static_cast<char *>(ws);
  const DevMeta m = meta_at(p, reinterpret_cast<const int32_t *>(base + L.meta));
  const int kind = mode == EB_MODE_DECODE ? 0 : (mode == EB_MODE_PREFILL ? 1 : 2);
  hipError_t e = launch_attention(h->shape, static_cast<const uint16_t *>(qkv), kv_of(kv), m,
                                  static_cast<uint16_t *>(out), reinterpret_cast<float *>(base + L.part_o),
                                  reinterpret_cast<float *>(base + L.part_ml), kind, st);
  return e == hipSuccess ? EB_OK : hip_fail(e, "attention");
}

eb_status eb_op_gather_kv(eb_handle *h, const eb_kv_cache *kv, const eb_batch *batch, void *out_k, void *out_v,
                          void *ws, size_t ws_bytes, void *stream) {
  eb_status s = check_kv(kv);
  if (s != EB_OK) return s;
  s = check_common(h, batch, EB_MODE_MIXED, kv->max_pages_per_seq);
  if (s != EB_OK) return s;
  if (batch->num_seqs == 0) return EB_OK;
  if (!out_k || !out_v) return fail(EB_ERR_NULL, "out_k or out_v is NULL");
  s = debug_check_tables(h, batch, kv, 1, static_cast<hipStream_t>(stream));
  if (s != EB_OK) return s;
  HostPlan p;
  build_plan(h->cfg, *batch, EB_MODE_MIXED, p);
  const WsLayout L = layout_for(h->shape, p, false);
  s = check_ws(ws, ws_bytes, L.total);
  if (s != EB_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = stage_meta(h, p, ws, L, st);
  if (s != EB_OK) return s;
  const DevMeta m = meta_at(p, reinterpret_cast<const int32_t *>(static_cast<char *>(ws) + L.meta));
  hipError_t e = launch_gather_kv(h->shape, kv_of(kv), m, static_cast<uint16_t *>(out_k),
                                  static_cast<uint16_t *>(out_v), st);
  return e == hipSuccess ? EB_OK : hip_fail(e, "gather");
}

}  // extern "C"
