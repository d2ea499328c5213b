/*
 * eb_layer.h — C ABI of libeb.so: one transformer decoder-layer step over a
 * token batch on an MI355X (gfx950), in exclusive-decode, exclusive-prefill
 * and mixed batch modes.
 *
 * What a step is.  The paper prices one iteration of the serving loop as
 * T_iter = alpha + beta * n_tok over a batch of n_tok rows whose decode share
 * is r = n_decode / n_tok (Sec. 1); exclusive batching runs prefill and decode
 * rows in separate iterations, mixed batching puts them in one (Sec. 1,
 * Sec. 3.1 "Timing Model").  Requests keep their KV cache between iterations
 * (Sec. 3.1 "System Model"), every iteration handles at most B rows under
 * chunked prefill (App. A.1), and the cache is paged (Sec. 4.1
 * "Implementation").  A decode request streams its whole cached context in
 * attention (App. A.2, "Effect of decode context length").  One call here is
 * one layer of such an iteration: for every request i with c_i tokens already
 * cached and n_i new rows,
 *
 *   a = RMSNorm(x) g1;  q,k,v = a Wqkv^T;  RoPE(q,k) at pos = c_i + j;
 *   append k,v (bf16) at pos;  o = causal GQA attention over keys 0..pos;
 *   h1 = x + o Wo^T;  m = SiLU(RMSNorm(h1) g2 Wg^T) * (RMSNorm(h1) g2 Wu^T);
 *   y = h1 + m Wd^T.
 *
 * Conventions shared by every entry point.
 *  - bf16 data are passed as raw 16-bit patterns (uint16 storage), row-major,
 *    contiguous.  Arithmetic is fp32 with bf16 inputs and outputs.
 *  - Pointers named *_host are host memory; every other data pointer is
 *    device memory of the current HIP device.  The caller owns all memory.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).  Calls
 *    only enqueue work on it and return without waiting; buffers must stay
 *    alive until the stream has finished the work.
 *  - Every argument check runs before anything is enqueued: a return of
 *    EB_ERR_NULL, EB_ERR_CONFIG, EB_ERR_BATCH, EB_ERR_MODE, EB_ERR_PAGES,
 *    EB_ERR_WORKSPACE or EB_ERR_LIMITS means no work was launched and no byte
 *    of device memory was written.  EB_ERR_HIP is different: a HIP call
 *    failed after the checks, possibly after earlier stages (the metadata
 *    copy, earlier kernels) were already enqueued on the stream; the
 *    outputs, the workspace and the new cache slots are then undefined
 *    (every other cache byte is still unchanged: no kernel writes outside
 *    the new slots).  The message for the last failure on the calling thread
 *    is eb_last_error().
 *  - Device block tables are not read back on the host in normal operation:
 *    eb_validate checks their contents from a host copy.  A handle created
 *    while the environment variable EB_DEBUG_VALIDATE is set (to anything
 *    but "0"), or by a library built with -DEB_DEBUG_VALIDATE, runs the
 *    same check inside every call that takes a cache: it copies the needed
 *    block-table rows to the host on the caller's stream, waits for them
 *    (a host synchronisation: debugging only) and returns EB_ERR_PAGES
 *    before enqueuing any work if an id is outside [0, num_pages) or a page
 *    is used twice.  Without it a bad id reads as zeros (kernels bound every
 *    page id by num_pages) and results are undefined, but no memory outside
 *    the cache is touched.
 *  - Supported shapes: head_dim in {64, 128}; n_q_heads a multiple of
 *    n_kv_heads with n_q_heads / n_kv_heads in {1, 2, 4, 8}; page_size 16;
 *    hidden and ffn multiples of 8.  Anything else is EB_ERR_CONFIG.
 *  - A handle is not thread-safe; separate handles are independent.
 */
#ifndef EB_LAYER_H
#define EB_LAYER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum eb_status {
  EB_OK = 0,
  EB_ERR_NULL = -1,      /* a required pointer is NULL */
  EB_ERR_CONFIG = -2,    /* unsupported layer shape */
  EB_ERR_BATCH = -3,     /* lengths inconsistent (n_i = 0, sum n_i != num_tokens, negative c_i, ...) */
  EB_ERR_MODE = -4,      /* batch not allowed by the entry point's mode */
  EB_ERR_PAGES = -5,     /* block table too short or holding ids outside [0, num_pages) or shared */
  EB_ERR_WORKSPACE = -6, /* workspace NULL or smaller than eb_workspace_bytes() */
  EB_ERR_LIMITS = -7,    /* batch larger than the handle was created for */
  EB_ERR_HIP = -8        /* a HIP runtime call or kernel launch failed */
} eb_status;

typedef enum eb_mode {
  EB_MODE_DECODE = 0,  /* exclusive decode: every n_i == 1 */
  EB_MODE_PREFILL = 1, /* exclusive prefill: every n_i >= 1, any c_i */
  EB_MODE_MIXED = 2    /* mixed: any n_i >= 1, decode and prefill rows in one step */
} eb_mode;

typedef enum eb_epilogue {
  EB_EPI_STORE = 0,    /* out = bf16(A W^T) */
  EB_EPI_RESIDUAL = 1, /* out = bf16(A W^T + residual) */
  EB_EPI_SILU_MUL = 2  /* W holds [gate; up] (2F rows): out[:, f] = bf16(SiLU(g_f) * u_f), F = N / 2 */
} eb_epilogue;

/* Layer shape.  rms_eps: RMSNorm epsilon; rope_theta: RoPE base.
 * n_experts > 0 makes the feed-forward part the mixture-of-experts block of
 * eb_op_moe_ffn (top_k experts per token, expert SwiGLU width expert_ffn,
 * renormalised weights unless moe_renormalize is 0; ffn is then unused and
 * may be 0); n_experts = 0 (a zero-initialised tail) is the dense SwiGLU of
 * width ffn.  qk_norm != 0 (the Qwen3 attention block): every q and k head of
 * the QKV projection is RMS-normalised over its head_dim values (epsilon
 * rms_eps, fp32) and multiplied by the gain q_norm or k_norm before RoPE;
 * 0 (a zero-initialised tail): no such norm. */
typedef struct eb_layer_config {
  int32_t hidden, n_q_heads, n_kv_heads, head_dim, ffn, page_size;
  float rms_eps, rope_theta;
  int32_t n_experts, top_k, expert_ffn, moe_renormalize;
  int32_t qk_norm;
} eb_layer_config;

/* Element type of the four projection matrices. */
typedef enum {
  EB_W_BF16 = 0,     /* bf16 values */
  EB_W_FP8_E4M3 = 1  /* 8-bit OCP E4M3 codes with one fp32 scale per output row */
} eb_weight_dtype;

/* Device pointers to the weights in the [out, in] layout:
 *   attn_norm, mlp_norm  [hidden] (bf16 always)
 *   w_qkv     [(n_q + 2 n_kv) head_dim, hidden], rows q heads, k heads, v heads
 *   w_o       [hidden, n_q head_dim]
 *   w_gate_up [2 ffn, hidden], rows gate then up
 *   w_down    [hidden, ffn]
 * w_dtype EB_W_BF16 (a zero-initialised struct): the projections hold bf16.
 * EB_W_FP8_E4M3: they hold E4M3 codes (one byte each, same layout) and
 * s_qkv, s_o, s_gate_up, s_down point to fp32 scales, one per row of the
 * matching matrix; the weight a code stands for is decode(code) * scale of
 * its row (the E4M3 values convert exactly to bf16 for the products, the
 * scale multiplies the fp32 sum).  A NaN code (0x7F, 0xFF) is the caller's
 * to avoid.  The scale pointers are ignored for bf16 weights. */
typedef struct eb_layer_weights {
  const void *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
  int32_t w_dtype;
  const float *s_qkv, *s_o, *s_gate_up, *s_down;
  /* mixture-of-experts layers (n_experts > 0; bf16 weights only, w_gate_up
   * and w_down unused): router [E, hidden], experts' gate/up
   * [E, 2 expert_ffn, hidden] (per expert gate rows, then up rows) and down
   * [E, hidden, expert_ffn] */
  const void *w_router, *w_experts_gate_up, *w_experts_down;
  /* per-head q and k norm gains, bf16 [head_dim] each (qk_norm layers;
   * unused otherwise) */
  const void *q_norm, *k_norm;
  /* optional fragment-packed copies of the four bf16 projections
   * (eb_pack_weight; NULL: none).  The weight-streaming GEMMs (steps of at
   * most 256 rows) read a packed copy instead of the row-major matrix, the
   * same values in the same order, so outputs are bitwise unchanged; the
   * 256 x 256 tiled GEMMs always read the row-major matrices, which stay
   * required.  Ignored for 8-bit weights and for a matrix whose shape
   * eb_packed_weight_bytes rejects.  A packed copy must be made from the
   * matrix it stands beside; the library cannot check that. */
  const void *p_qkv, *p_o, *p_gate_up, *p_down;
} eb_layer_weights;

/* Element type of the KV cache. */
typedef enum {
  EB_KV_BF16 = 0,     /* bf16 values */
  EB_KV_FP8_E4M3 = 1  /* 8-bit codes, OCP E4M3 (bias 7, no infinity, 0x7F/0xFF NaN, largest finite 448) */
} eb_kv_dtype;

/* Paged KV cache (device).  k_cache, v_cache: [num_pages, n_kv_heads,
 * page_size, head_dim] elements of kv_dtype.  block_tables: int32
 * [num_seqs, max_pages_per_seq]; logical page j of request i is physical
 * page block_tables[i][j].  Entries past a request's last needed page are
 * never read.  The library never allocates or frees pages.
 *
 * An 8-bit cache halves the bytes a decode step streams (decode attention
 * reads every cached position of every decode request: Sec. 1, App. A.2).
 * A cached code stands for decode(code) * scale (k_scale for keys, v_scale
 * for values); the step stores e4m3(bf16(x) / scale), the division rounded in
 * fp32, nearest-even, saturated to +-448 (NaN keeps its sign: 0x7F / 0xFF).
 * Scales must be finite and positive for EB_KV_FP8_E4M3 and are ignored for
 * bf16; a zero-initialised struct is a bf16 cache. */
typedef struct eb_kv_cache {
  void *k_cache, *v_cache;
  int32_t num_pages;
  const int32_t *block_tables;
  int32_t max_pages_per_seq;
  int32_t kv_dtype; /* eb_kv_dtype */
  float k_scale, v_scale;
} eb_kv_cache;

/* One step's requests.  context_lens_host[i] = c_i, tokens already cached
 * before the step; chunk_lens_host[i] = n_i >= 1, new rows.  Rows of request
 * i are x rows off_i .. off_i + n_i - 1 with off_i = n_0 + ... + n_{i-1}.
 * num_tokens must equal the sum of n_i.  Both arrays are HOST memory. */
typedef struct eb_batch {
  int32_t num_seqs, num_tokens;
  const int32_t *context_lens_host, *chunk_lens_host;
} eb_batch;

typedef struct eb_handle eb_handle;

/* Create a handle for one layer shape on the current HIP device, sized for at
 * most max_seqs requests and max_tokens rows per step.  Allocates small
 * pinned host staging buffers.  Errors: EB_ERR_NULL, EB_ERR_CONFIG,
 * EB_ERR_LIMITS (max_seqs or max_tokens < 1), EB_ERR_HIP. */
eb_status eb_create(const eb_layer_config *cfg, int32_t max_seqs, int32_t max_tokens, eb_handle **out);

/* Release a handle (waits for nothing: the caller synchronises first). */
void eb_destroy(eb_handle *h);

/* Bytes of device workspace a step over `batch` needs in `mode` (256-byte
 * aligned base required).  Returns 0 if the batch is invalid for the mode. */
size_t eb_workspace_bytes(const eb_handle *h, const eb_batch *batch, eb_mode mode);

/* Intermediate buffers of a layer step inside its workspace.  After a
 * step over `batch` in `mode` (or the last layer of a stack), the workspace
 * holds, at the byte offset eb_workspace_offset() returns:
 *   EB_WS_QKV  bf16 [num_tokens, (n_q + 2 n_kv) head_dim], the QKV projection
 *              output with the q heads normalised (qk_norm) and rotated in
 *              place, k and v as projected (the cache holds rotated k)
 *   EB_WS_ATTN bf16 [num_tokens, n_q head_dim], the attention output
 *   EB_WS_H1   bf16 [num_tokens, hidden], h1 = x + attn Wo^T
 *   EB_WS_MLP  bf16 [num_tokens, ffn], m = SiLU(b Wg^T) * (b Wu^T) (dense
 *              layers only)
 *   EB_WS_NORM bf16 [num_tokens, hidden], b = RMSNorm(h1) g2
 * The residual stream dominates y (|x| is far above |attn Wo^T| at these
 * weight scales), so attention errors are visible only in these buffers;
 * they exist for stage-level parity tests.  Returns (size_t)-1 for an
 * invalid or empty batch, an unknown buffer, or EB_WS_MLP of an MoE layer. */
typedef enum eb_ws_buffer {
  EB_WS_QKV = 0,
  EB_WS_ATTN = 1,
  EB_WS_H1 = 2,
  EB_WS_MLP = 3,
  EB_WS_NORM = 4
} eb_ws_buffer;
size_t eb_workspace_offset(const eb_handle *h, const eb_batch *batch, eb_mode mode, int32_t which);

/* The three step entry points.  x: bf16 [num_tokens, hidden] (input rows),
 * y: bf16 [num_tokens, hidden] (output; must not alias x).  Writes y, the
 * workspace and exactly the cache slots of positions c_i .. c_i + n_i - 1;
 * every other cache byte is left unchanged.  The block-table pages for all
 * positions < c_i + n_i must exist (checked on the host by eb_validate;
 * device block tables are not read back here).
 *   decode : every n_i == 1 (EB_ERR_MODE otherwise)
 *   prefill: any n_i >= 1
 *   mixed  : any n_i >= 1; decode and prefill attention share one launch. */
eb_status eb_layer_step_decode(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv,
                               const eb_batch *batch, const void *x, void *y, void *ws, size_t ws_bytes,
                               void *stream);
eb_status eb_layer_step_prefill(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv,
                                const eb_batch *batch, const void *x, void *y, void *ws, size_t ws_bytes,
                                void *stream);
eb_status eb_layer_step_mixed(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv,
                              const eb_batch *batch, const void *x, void *y, void *ws, size_t ws_bytes,
                              void *stream);

/* eb_layer_step_mixed without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The step's intermediate buffers live
 * in a fixed scratch array inside the library, eb_noalloc_scratch_bytes()
 * = 64 MiB per GPU, held from the library's first use on a GPU until the
 * process ends (its address is looked up once per device in eb_create).
 * The call allocates no device or pinned memory (the handle's staging
 * buffers come from eb_create; the host planner uses ordinary heap memory)
 * and never profiles.  Same arguments, modes, checks and results as
 * eb_layer_step_mixed, bitwise; EB_ERR_WORKSPACE when the batch needs more
 * than the scratch holds (eb_workspace_bytes(h, batch, EB_MODE_MIXED) >
 * eb_noalloc_scratch_bytes()), EB_ERR_HIP if the scratch's address could not
 * be found.  Every call on one GPU shares that GPU's scratch and leaves its
 * contents behind (no kernel of the step reads a scratch byte it did not
 * write in the same call, so nothing needs clearing): calls that may overlap
 * on one GPU (other streams, other handles or threads) race and must be
 * serialised by the caller. */
size_t eb_noalloc_scratch_bytes(void);
eb_status eb_layer_step_mixed_noalloc(eb_handle *h, const eb_layer_weights *w, const eb_kv_cache *kv,
                                      const eb_batch *batch, const void *x, void *y, void *stream);

/* A model step: n_layers decoder layers over one batch.  The paper's
 * iteration time is that of the whole model over the batch (Sec. 1,
 * Sec. 3.1 "Timing Model"); every layer sees the same requests and rows.
 * Layer l maps its input (x for l = 0, layer l - 1's output otherwise) to
 * its output with weights[l] and kv[l]; layer n_layers - 1 writes y (which
 * must not alias x).  weights and kv are HOST arrays of n_layers structs;
 * kv entries may name the same cache arrays, in which case each layer
 * writes the new positions' slots in turn and attends over its own values
 * (it appends before it attends).  The batch is planned and its metadata
 * staged once for all layers.  mode is one of the three step modes, with the
 * same batch constraints as the layer entry points.  ws must hold
 * eb_stack_workspace_bytes() bytes (one layer's workspace plus one
 * activation buffer that alternates with y).  With profiling on,
 * eb_profile_read() returns each stage's time summed over the layers.
 * Errors as for the layer steps, plus EB_ERR_CONFIG for n_layers < 1 and
 * EB_ERR_MODE for an unknown mode; a failing layer is named in the message. */
size_t eb_stack_workspace_bytes(const eb_handle *h, const eb_batch *batch, eb_mode mode);
eb_status eb_stack_step(eb_handle *h, eb_mode mode, int32_t n_layers, const eb_layer_weights *weights,
                        const eb_kv_cache *kv, const eb_batch *batch, const void *x, void *y, void *ws,
                        size_t ws_bytes, void *stream);

/* Host-only check of a step's inputs (no GPU needed): shape support, lengths,
 * mode constraints, and block-table contents (ids in [0, num_pages) for every
 * needed logical page, no physical page used twice).  block_tables_host is
 * int32 [num_seqs, max_pages_per_seq] in host memory. */
eb_status eb_validate(const eb_layer_config *cfg, const eb_batch *batch, const int32_t *block_tables_host,
                      int32_t num_pages, int32_t max_pages_per_seq, eb_mode mode);

/* Per-stage timing.  eb_profile(h, n, mask) with n >= 1 makes every
 * following step on h record HIP events around the stages whose bit is set
 * in mask (bit i: stage i; 0: every stage) on its stream (a marker per stage
 * boundary, a few microseconds of host time each, no synchronisation), into
 * a ring of n step slots created by this call; n = 0 switches it off.
 * eb_profile_read() waits for the recorded steps and writes into ms[] (host)
 * the duration in ms of up to `cap` stages, in launch order, averaged over
 * the recorded steps (the last n of them), each a sum over the step's layers
 * (stages outside the mask read 0); it returns how many it wrote (0 if no
 * profiled step has run since eb_profile, -1 on a HIP error).  Stage names:
 * eb_profile_stage_name(i) (NULL past the last).  Stages a step does not need
 * read 0.  EB_ERR_CONFIG for n < 0 or a mask bit past the last stage. */
eb_status eb_profile(eb_handle *h, int32_t steps, uint32_t stage_mask);
int32_t eb_profile_read(eb_handle *h, float *ms, int32_t cap);
const char *eb_profile_stage_name(int32_t i);

const char *eb_status_str(eb_status s);
const char *eb_last_error(void); /* thread-local message of the last failure */

/* ---- single operations of the step, same conventions (for parity tests) ---- */

/* out[r] = bf16(x[r] / sqrt(mean(x[r]^2) + eps) * gamma), rows x hidden.
 * The pre-attention and pre-MLP norms of the layer (the per-token "other"
 * work of the step, App. A.2 "Kernel breakdown"). */
eb_status eb_op_rmsnorm(const eb_handle *h, const void *x, const void *gamma, void *out, int32_t rows,
                        void *stream);

/* The projection GEMMs of the step: the QKV, O, gate/up and down products
 * that make up the 24 d^2 FLOPs per token of prefill (App. A.1) and do not
 * change with the decode share or the context (App. A.2).
 * out = epilogue(A W^T): A bf16 [M, K], W bf16 [N, K], out bf16 [M, N] (or
 * [M, N/2] for EB_EPI_SILU_MUL), residual bf16 [M, N] (EB_EPI_RESIDUAL only).
 * N and K must be multiples of 8 (EB_ERR_CONFIG otherwise).
 * ws: device scratch of at least eb_op_gemm_workspace_bytes(M, N, K). */
size_t eb_op_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K);
eb_status eb_op_gemm(const void *A, const void *W, void *out, const void *residual, int32_t M, int32_t N,
                     int32_t K, eb_epilogue epi, void *ws, size_t ws_bytes, void *stream);

/* eb_op_gemm with 8-bit weights: W holds E4M3 codes [N, K] (one byte each)
 * and w_scale (device, fp32 [N], 16-byte aligned) one scale per row; the
 * product is out = epilogue(A (decode(W) * w_scale)^T), the scale applied to
 * each column's fp32 sum.  ws: at least eb_op_gemm_workspace_bytes(M, N, K),
 * which covers both weight types.  EB_ERR_LIMITS when no kernel reaches the
 * operands through its 32-bit buffer ranges: W of 2^31 bytes or more, or A
 * of 2^31 bytes or more unless K is a multiple of 64, M >= 256 and W is
 * under 2^30 bytes.  A NaN code (0x7F, 0xFF) is the caller's to avoid. */
/* Fragment-packed copy of a bf16 weight matrix W [rows, cols] (device, row
 * major) for the weight-streaming GEMMs: each 16-row x 32-column block of W
 * becomes one contiguous 1 KiB run in the lane order of the 16x16x32 bf16
 * matrix-core operand (lane l: row 16 g + l % 16, columns 32 c + 8 (l / 16)
 * .. + 7), block (g, c) at byte (g cols / 32 + c) 1024, so that one 16-byte
 * load per lane fills an operand register from 1 KiB of contiguous memory.
 * Made once per matrix (weights are fixed while serving, Sec. 4.1), outside
 * the steps.  eb_packed_weight_bytes returns the size of the copy (rows cols
 * 2), or 0 when the shape has no packed form (rows % 16, cols % 32 nonzero,
 * or 2 rows cols >= 2^31).  eb_pack_weight writes it into `packed`
 * (caller-owned device memory of that size, not overlapping W), enqueued on
 * `stream`; EB_ERR_NULL for a null pointer, EB_ERR_CONFIG for a shape
 * without a packed form, EB_ERR_HIP if the launch fails.  The split SwiGLU matrix [2 ffn, hidden]
 * additionally needs ffn % 16 == 0 for its packed copy to be read. */
size_t eb_packed_weight_bytes(int rows, int cols);
eb_status eb_pack_weight(const void *w, void *packed, int rows, int cols, void *stream);

eb_status eb_op_gemm_w8(const void *A, const void *W, const float *w_scale, void *out, const void *residual,
                        int32_t M, int32_t N, int32_t K, eb_epilogue epi, void *ws, size_t ws_bytes, void *stream);

/* Mixture-of-experts feed-forward block (the paper's MoE model, Qwen3-30B-A3B,
 * Sec. 4.1 "Models"; its routing and expert work dominate that model's step,
 * App. A.2 "Kernel breakdown"), in place of the dense SwiGLU:
 *   logits[t] = b[t] W_r^T, fp32 sums of the bf16 products, kept in fp32
 *   S(t)      = the top_k largest logits of token t (equal logits: lower expert)
 *   w[t, e]   = exp(logits[t, e] - max_t) / (sum of the same over S(t) when
 *               renormalize, over all E experts otherwise), e in S(t)
 *   m         = SiLU(b[t] Wg_e^T) * (b[t] Wu_e^T), rounded to bf16
 *   out[t]    = bf16(residual[t] + sum_{e in S(t)} w[t, e] * (m Wd_e^T))
 * b bf16 [T, d] (the block's normalised input), residual bf16 [T, d] or NULL,
 * w_router bf16 [E, d], w_gate_up bf16 [E, 2F, d] (per expert: F gate rows,
 * then F up rows), w_down bf16 [E, d, F], out bf16 [T, d]; all device memory,
 * caller-owned.  ids_out (int32 [T, top_k]) and weights_out (fp32 [T, top_k]),
 * when not NULL, receive each token's experts (largest logit first) and
 * weights.  Requires d % 32 == 0, F % 8 == 0, E % 16 == 0 and E <= 256,
 * 1 <= top_k <= min(E, 64) (EB_ERR_CONFIG); operands within the kernels'
 * 32-bit ranges (EB_ERR_LIMITS).  NaN inputs are the caller's to avoid.
 * ws: device scratch of at least eb_op_moe_ffn_workspace_bytes(...). */
size_t eb_op_moe_ffn_workspace_bytes(int32_t T, int32_t d, int32_t E, int32_t top_k, int32_t F);
eb_status eb_op_moe_ffn(const void *b, const void *residual, const void *w_router, const void *w_gate_up,
                        const void *w_down, int32_t T, int32_t d, int32_t E, int32_t top_k, int32_t F,
                        int32_t renormalize, void *out, int32_t *ids_out, float *weights_out, void *ws,
                        size_t ws_bytes, void *stream);

/* The cache append of the step: new keys and values join each request's
 * paged KV cache, which the paper's engine keeps unchanged across
 * iterations (Sec. 3.1 "System Model", Sec. 4.1 "Implementation").
 * RoPE on the q and k heads of qkv (bf16 [num_tokens, (n_q + 2 n_kv) head_dim],
 * the QKV projection output) at pos = c_i + j; q is rotated in place, the
 * rotated k and the v heads are written to the cache.  A handle whose config
 * has qk_norm set gets EB_ERR_CONFIG: this entry has no norm gains (the layer
 * step entry points apply the norms). */
eb_status eb_op_rope_kv_append(eb_handle *h, void *qkv, const eb_kv_cache *kv, const eb_batch *batch,
                               void *ws, size_t ws_bytes, void *stream);

/* Attention of the step: decode rows stream their whole cached context
 * (memory bound, App. A.2 "Effect of decode context length"), prefill rows
 * are causal over their prefix and chunk (compute bound, App. A.1), and the
 * mixed plan runs both kinds in one launch, the kernel in which the paper
 * locates mixed-batch interference (Sec. 1, Fig. kernel_breakdown).
 * Attention of every row over keys 0..pos of its request, reading rotated q
 * from qkv and keys/values from the cache (already appended); out bf16
 * [num_tokens, n_q head_dim].  mode selects the launch plan exactly as the
 * step entry points do. */
eb_status eb_op_attention(eb_handle *h, const void *qkv, const eb_kv_cache *kv, const eb_batch *batch,
                          void *out, void *ws, size_t ws_bytes, eb_mode mode, void *stream);

/* The paging of the cache (Sec. 4.1 "Implementation": paged attention left
 * unchanged) as a plain copy, for bit-exact checks of the block-table
 * addressing every attention kernel uses.
 * Dense copy of every request's cached positions 0 .. c_i + n_i - 1 through
 * its block table: out_k, out_v [sum_i (c_i + n_i), n_kv_heads, head_dim]
 * elements of the cache's type (bf16, or the raw 8-bit codes), requests in
 * order.  Pure paging: bit-exact. */
eb_status eb_op_gather_kv(eb_handle *h, const eb_kv_cache *kv, const eb_batch *batch, void *out_k,
                          void *out_v, void *ws, size_t ws_bytes, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* EB_LAYER_H */
