// Mixture-of-experts feed-forward block: routing, the expert-sorted order and
// the weighted combine (the expert products are the grouped GEMM kernel).
//
//   logits[t] = b[t] W_r^T (fp32 sums of bf16 products, kept in fp32)
//   S(t)      = the k largest logits (equal logits: lower expert first)
//   w[t, e]   = exp(logits[t, e] - max) over S(t), divided by its sum over
//               S(t) (renormalised) or over all E experts
//   out[t]    = bf16(residual[t] + sum_j w[t, j] y[t, j])
//
// with y[t, j] the fp32 output of expert S(t)_j for token t.
#include "device_common.h"
#include "eb_internal.h"

namespace eb {

constexpr int kMoeTokens = 16;  // tokens per logits wavefront

// Logits: one wavefront per 16 tokens x 16 experts, the 16x16x32 MFMA with
// the experts as rows and the tokens as columns, both operands read straight
// from global memory (W_r is shared by every wave and stays in L2), eight
// K steps of loads issued before their products.  fp32 out [T, E].
__global__ __launch_bounds__(64) void k_moe_logits(const uint16_t *__restrict__ b, const uint16_t *__restrict__ wr,
                                                   int T, int d, int E, float *__restrict__ logits) {
  const int lane = threadIdx.x;
  const int t0 = blockIdx.x * kMoeTokens, e0 = blockIdx.y * 16;
  const int lr = lane & 15, lgp = lane >> 4;
  const buf_rsrc_t rb = make_rsrc(b, (int)min((size_t)T * d * 2, (size_t)0x7FFFFFFF));
  const buf_rsrc_t rr = make_rsrc(wr, (int)min((size_t)E * d * 2, (size_t)0x7FFFFFFF));
  const int tok = t0 + lr;
  const uint32_t boff = tok < T ? ((uint32_t)tok * (uint32_t)d + 8u * lgp) * 2u : 0x80000000u;
  const uint32_t woff = ((uint32_t)(e0 + lr) * (uint32_t)d + 8u * lgp) * 2u;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  constexpr int U = 8;
  for (int kk = 0; kk < d; kk += 32 * U) {
    u32x4_t wf[U], bf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kk + 32 * u;
      const bool ok = k < d;
      wf[u] = buf_ld_u32x4<0>(rr, (int)(ok ? woff + 2u * k : 0x80000000u));
      bf[u] = buf_ld_u32x4<0>(rb, (int)(ok && boff != 0x80000000u ? boff + 2u * k : 0x80000000u));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc = mfma16x16x32(wf[u], bf[u], acc);
  }
  // lane holds experts e0 + 4 lgp .. + 3 of token lr
  if (tok < T) *reinterpret_cast<f32x4_t *>(logits + (size_t)tok * E + e0 + 4 * lgp) = acc;
}

// Top k of each token's logits: one wavefront per token, k rounds of a
// wave-wide arg-max (equal values: lower expert), then the weights.
__global__ __launch_bounds__(256) void k_moe_topk(const float *__restrict__ logits, int T, int E, int k,
                                                  int renormalize, int32_t *__restrict__ ids,
                                                  float *__restrict__ wts) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float *row = logits + (size_t)t * E;
  float v[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = lane + 64 * c < E ? row[lane + 64 * c] : -INFINITY;
  float sel_v = 0.f, top = 0.f, sum_sel = 0.f;
  int sel_e = 0;
  for (int j = 0; j < k; ++j) {
    // this lane's best (value, lowest expert), then the wave's
    float bv = v[0];
    int be = lane;
#pragma unroll
    for (int c = 1; c < 4; ++c)
      if (v[c] > bv) {
        bv = v[c];
        be = lane + 64 * c;
      }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off, 64);
      const int oe = __shfl_xor(be, off, 64);
      if (ov > bv || (ov == bv && oe < be)) {
        bv = ov;
        be = oe;
      }
    }
    if (j == 0) top = bv;
    const float p = __expf(bv - top);
    sum_sel += p;
    if (lane == j) {
      sel_v = p;
      sel_e = be;
    }
    // the owner takes the chosen value out
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (lane + 64 * c == be) v[c] = -INFINITY;
  }
  float denom = sum_sel;
  if (!renormalize) {  // the softmax over all E experts (top is the largest logit)
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (lane + 64 * c < E) s += __expf(row[lane + 64 * c] - top);
    denom = wave_sum(s);
  }
  if (lane < k) {
    ids[(size_t)t * k + lane] = sel_e;
    wts[(size_t)t * k + lane] = sel_v / denom;
  }
}

// One block: expert counts, their offsets in the sorted order, the row
// tiles (up to tile_rows rows of one expert) and each assignment's sorted
// position.
// Positions within an expert follow the order of the block's atomics; every
// later step is independent of that order (rows are independent in the
// products and the combine reads the slots in token order).
__global__ __launch_bounds__(1024) void k_moe_plan(const int32_t *__restrict__ ids, int P, int E, int k,
                                                   int tile_rows, int max_tiles, int32_t *__restrict__ offsets,
                                                   int32_t *__restrict__ sorted_tok, int32_t *__restrict__ pos_of,
                                                   int32_t *__restrict__ tiles, int32_t *__restrict__ n_tiles) {
  __shared__ int cnt[256], cur[256], toff[257];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += blockDim.x) cnt[e] = 0;
  __syncthreads();
  // (ids come from the routing kernel; clamped all the same, so that no
  // input can steer a write outside the tables)
  auto expert = [&](int i) { return min(max(ids[i], 0), E - 1); };
  for (int i = tid; i < P; i += blockDim.x) atomicAdd(&cnt[expert(i)], 1);
  __syncthreads();
  if (tid == 0) {
    int o = 0, to = 0;
    for (int e = 0; e < E; ++e) {
      offsets[e] = o;
      cur[e] = o;
      toff[e] = to;
      o += cnt[e];
      to += (cnt[e] + tile_rows - 1) / tile_rows;
    }
    offsets[E] = o;
    toff[E] = to;
    *n_tiles = min(to, max_tiles);
  }
  __syncthreads();
  for (int e = tid; e < E; e += blockDim.x) {
    const int n = cnt[e], base = cur[e];
    for (int j = 0, r = toff[e]; j < n && r < max_tiles; j += tile_rows, ++r) {
      tiles[r] = e;
      tiles[max_tiles + r] = base + j;
      tiles[2 * max_tiles + r] = min(tile_rows, n - j);
    }
  }
  __syncthreads();
  for (int i = tid; i < P; i += blockDim.x) {
    const int p = atomicAdd(&cur[expert(i)], 1);
    sorted_tok[p] = i / k;
    pos_of[i] = p;
  }
}

// out[t] = bf16(res[t] + sum_j w[t, j] y[pos_of[t k + j]]): one block per
// token, four columns per thread and step.
__global__ __launch_bounds__(256) void k_moe_combine(const float *__restrict__ y, const int32_t *__restrict__ pos_of,
                                                     const float *__restrict__ wts, const uint16_t *__restrict__ res,
                                                     uint16_t *__restrict__ out, int d, int k) {
  const int t = blockIdx.x;
  for (int c = 4 * threadIdx.x; c < d; c += 4 * blockDim.x) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float w = wts[(size_t)t * k + j];
      const f32x4_t v = *reinterpret_cast<const f32x4_t *>(y + (size_t)pos_of[(size_t)t * k + j] * d + c);
      acc += w * v;
    }
    if (res) {
      const u32x2_t r = *reinterpret_cast<const u32x2_t *>(res + (size_t)t * d + c);
      acc[0] += bf16_lo(r[0]);
      acc[1] += bf16_hi(r[0]);
      acc[2] += bf16_lo(r[1]);
      acc[3] += bf16_hi(r[1]);
    }
    *reinterpret_cast<u32x2_t *>(out + (size_t)t * d + c) =
        u32x2_t{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3])};
  }
}

hipError_t launch_moe_route(const uint16_t *b, const uint16_t *wr, int T, int d, int E, int k, int renormalize,
                            float *logits, int32_t *ids, float *wts, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_moe_logits, dim3((T + kMoeTokens - 1) / kMoeTokens, E / 16), dim3(64), 0, st, b, wr, T, d, E,
                     logits);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_moe_topk, dim3((T + 3) / 4), dim3(256), 0, st, logits, T, E, k, renormalize, ids, wts);
  return hipGetLastError();
}

hipError_t launch_moe_plan(const int32_t *ids, int P, int E, int k, int tile_rows, int max_tiles, int32_t *offsets,
                           int32_t *sorted_tok, int32_t *pos_of, int32_t *tiles, int32_t *n_tiles, hipStream_t st) {
  hipLaunchKernelGGL(k_moe_plan, dim3(1), dim3(1024), 0, st, ids, P, E, k, tile_rows, max_tiles, offsets, sorted_tok,
                     pos_of, tiles, n_tiles);
  return hipGetLastError();
}

hipError_t launch_moe_combine(const float *y, const int32_t *pos_of, const float *wts, const uint16_t *res,
                              uint16_t *out, int T, int d, int k, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_moe_combine, dim3(T), dim3(256), 0, st, y, pos_of, wts, res, out, d, k);
  return hipGetLastError();
}

}  // namespace eb
