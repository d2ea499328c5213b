// RMSNorm, RoPE + paged KV append, and the dense KV gather probe.
#include "device_common.h"
#include "eb_internal.h"

namespace eb {

// ---------------------------------------------------------------------------
// RMSNorm: out = bf16(x / sqrt(mean(x^2) + eps) * gamma).  One wavefront per
// row, 16-byte accesses.  Rows of up to 64 * 8 * MAXC elements stay in
// registers: every load of the row and of gamma is issued before the first
// use, so the kernel waits for memory once; longer rows take a second pass.
// ---------------------------------------------------------------------------
// MC: 16-byte chunks per lane held in registers (rows up to 512 MC wide),
// the smallest of 4, 8, 16 that holds the row, so that narrow rows leave
// room for more waves
template <int MC>
__global__ __launch_bounds__(256) void k_rmsnorm(const uint16_t *__restrict__ x, const uint16_t *__restrict__ g,
                                                 uint16_t *__restrict__ out, int rows, int d, float eps) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const uint16_t *xr = x + (size_t)row * d;
  uint16_t *orow = out + (size_t)row * d;
  const int nch = d >> 3;
  if (nch <= 64 * MC) {
    u32x4_t v[MC], gv[MC];
#pragma unroll
    for (int j = 0; j < MC; ++j) {
      const int c = lane + 64 * j;
      v[j] = c < nch ? ld_u32x4(xr + c * 8) : u32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < MC; ++j) {
      const int c = lane + 64 * j;
      gv[j] = c < nch ? ld_u32x4(g + c * 8) : u32x4_t{0u, 0u, 0u, 0u};  // shared by all rows: an L2 hit
    }
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < MC; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a = bf16_lo(v[j][i]), b = bf16_hi(v[j][i]);
        ss += a * a + b * b;
      }
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int j = 0; j < MC; ++j) {
      const int c = lane + 64 * j;
      if (c < nch) {
        u32x4_t o;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[i] = pack_bf16x2(bf16_lo(v[j][i]) * inv * bf16_lo(gv[j][i]), bf16_hi(v[j][i]) * inv * bf16_hi(gv[j][i]));
        st_u32x4(orow + c * 8, o);
      }
    }
    return;
  }
  float ss = 0.f;
  for (int c = lane; c < nch; c += 64) {
    u32x4_t v = ld_u32x4(xr + c * 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float a = bf16_lo(v[i]), b = bf16_hi(v[i]);
      ss += a * a + b * b;
    }
  }
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = lane; c < nch; c += 64) {
    u32x4_t v = ld_u32x4(xr + c * 8);
    u32x4_t gv = ld_u32x4(g + c * 8);
    u32x4_t o;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = pack_bf16x2(bf16_lo(v[i]) * inv * bf16_lo(gv[i]), bf16_hi(v[i]) * inv * bf16_hi(gv[i]));
    st_u32x4(orow + c * 8, o);
  }
}

hipError_t launch_rmsnorm(const uint16_t *x, const uint16_t *gamma, uint16_t *out, int rows, int d, float eps,
                          hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int nch = d >> 3;
  if (nch <= 64 * 4)
    hipLaunchKernelGGL(k_rmsnorm<4>, dim3((rows + 3) / 4), dim3(256), 0, st, x, gamma, out, rows, d, eps);
  else if (nch <= 64 * 8)
    hipLaunchKernelGGL(k_rmsnorm<8>, dim3((rows + 3) / 4), dim3(256), 0, st, x, gamma, out, rows, d, eps);
  else
    hipLaunchKernelGGL(k_rmsnorm<16>, dim3((rows + 3) / 4), dim3(256), 0, st, x, gamma, out, rows, d, eps);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RoPE (rotate-half pairs (t, t + hd/2), frequency theta^(-2t/hd), angle
// formed in fp64) on the q and k heads of one QKV row, q rotated in place,
// rotated k and v stored at the row's slot of its request's paged cache.
// Codes of eight bf16 values (packed pairs) divided by scale.
__device__ __forceinline__ u32x2_t e4m3x8_of_bf16x8(u32x4_t w, float scale) {
  u32x2_t r;
#pragma unroll
  for (int i = 0; i < 2; ++i)
    r[i] = e4m3x4_from_f32(bf16_lo(w[2 * i]) / scale, bf16_hi(w[2 * i]) / scale, bf16_lo(w[2 * i + 1]) / scale,
                           bf16_hi(w[2 * i + 1]) / scale);
  return r;
}

// One block per row; a thread moves 8 consecutive dims of one half of a
// head and their 8 partners in 16-byte accesses.  The angle pos * freq is
// formed and reduced to [-pi, pi] in fp64; its sine and cosine are then
// taken in fp32 (the reduced angle is small, so fp32 is accurate to an ulp).
// ---------------------------------------------------------------------------
// With an 8-bit cache (F8) the new K and V enter as codes of their bf16
// values divided by the scale (the division rounded in fp32).  With QKN each
// q and k head is first RMS-normalised over its hd values and scaled by its
// gain (gq for q heads, gk for k heads), in fp32, before the rotation.
// FUSED: the row first comes out of the QKV projection's split-K partials
// (fp32 [splits][T][cols], summed in split order) times the row scale of the
// RMSNorm that preceded the projection, 1 / sqrt(sum_s ssq[s][r] / d + eps)
// (the projection ran on x * gamma, see the weight-streaming GEMM's
// PRENORM form); it is rounded to bf16 into qkv and then rotated and
// appended as in the plain form.
struct QkvPartials {
  const float *part, *ssq;
  int splits, d;
  float eps;
};
template <bool F8, bool QKN, bool FUSED = false>
__global__ __launch_bounds__(256) void k_rope_append(uint16_t *__restrict__ qkv, uint16_t *__restrict__ kc,
                                                     uint16_t *__restrict__ vc, const int32_t *__restrict__ bt,
                                                     int num_pages, int max_pages, DevMeta m, int nq, int nkv,
                                                     int hd, double log2_theta, float ks, float vs,
                                                     const uint16_t *__restrict__ gq,
                                                     const uint16_t *__restrict__ gk, float eps,
                                                     QkvPartials qp = QkvPartials{}) {
  __shared__ float cs[64], sn[64];
  const int r = blockIdx.x;
  // block y of the row takes heads [h_lo, h_hi) of the q, k, v heads
  const int nh = nq + 2 * nkv;
  const int hpb = (nh + gridDim.y - 1) / gridDim.y;
  const int h_lo = blockIdx.y * hpb, h_hi = min(nh, h_lo + hpb);
  const int seq = m.row_seq[r];
  const int pos = m.row_pos[r];
  const int half = hd >> 1;
  // FUSED: the loads of the thread's first 4 columns (a block's heads fit
  // in one pass at 256 threads) are issued before the angle table is
  // formed, so the table's fp64 work runs under their latency; one barrier
  // then publishes both the table and the row
  const int cols_f = nh * hd;
  const size_t stride_f = (size_t)m.T * cols_f;
  const float *p0 = FUSED ? qp.part + (size_t)r * cols_f : nullptr;
  const int c_first = h_lo * hd + threadIdx.x * 4;
  f32x4_t x_first = {0.f, 0.f, 0.f, 0.f};
  float inv = 1.f;
  if constexpr (FUSED) {
    float ss = 0.f;
    for (int s = 0; s < qp.splits; ++s) ss += qp.ssq[(size_t)s * m.T + r];
    if (c_first < h_hi * hd)
      for (int s = 0; s < qp.splits; ++s) x_first += *reinterpret_cast<const f32x4_t *>(p0 + s * stride_f + c_first);
    inv = 1.0f / sqrtf(ss / (float)qp.d + qp.eps);
  }
  for (int t = threadIdx.x; t < half; t += blockDim.x) {
    const double inv_freq = exp2(-(2.0 * t / hd) * log2_theta);
    const double ang = (double)pos * inv_freq;
    const double two_pi = 6.283185307179586476925286766559;
    const double red = fma(-rint(ang / two_pi), two_pi, ang);
    float s, c;
    sincosf((float)red, &s, &c);
    cs[t] = c;
    sn[t] = s;
  }
  if constexpr (FUSED) {
    uint16_t *dst = qkv + (size_t)r * cols_f;
    for (int c = c_first; c < h_hi * hd; c += blockDim.x * 4) {
      f32x4_t x = x_first;
      if (c != c_first) {
        x = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < qp.splits; ++s) x += *reinterpret_cast<const f32x4_t *>(p0 + s * stride_f + c);
      }
      *reinterpret_cast<u32x2_t *>(dst + c) = u32x2_t{pack_bf16x2(x[0] * inv, x[1] * inv), pack_bf16x2(x[2] * inv, x[3] * inv)};
    }
  }
  __syncthreads();  // the angle table, and (FUSED) the row's bf16 values read back by other threads below
  const int cols = (nq + 2 * nkv) * hd;
  uint16_t *row = qkv + (size_t)r * cols;
  const int page = bt[(size_t)seq * max_pages + pos / kPageSize];
  const bool page_ok = page >= 0 && page < num_pages;
  const int slot = pos % kPageSize;
  const int hch = half / 8;  // 8-dim chunks per half head
  // q and k heads: (head, chunk of the first half) per thread
  const int hk_hi = min(h_hi, nq + nkv);
  const int items = h_lo < hk_hi ? (hk_hi - h_lo) * hch : 0;
  for (int i = threadIdx.x; i < items; i += blockDim.x) {
    const int h = h_lo + i / hch, t0 = (i % hch) * 8;
    const u32x4_t a = ld_u32x4(row + h * hd + t0);
    const u32x4_t b = ld_u32x4(row + h * hd + t0 + half);
    float fa[8], fb[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      fa[2 * e] = bf16_lo(a[e]);
      fa[2 * e + 1] = bf16_hi(a[e]);
      fb[2 * e] = bf16_lo(b[e]);
      fb[2 * e + 1] = bf16_hi(b[e]);
    }
    if constexpr (QKN) {
      // the hch threads of one head are adjacent lanes of one wavefront (hch
      // divides 64 and the thread count, items is a multiple of hch), all
      // active together: the head's sum of squares in log2(hch) exchanges
      float ss = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) ss += fa[e] * fa[e] + fb[e] * fb[e];
      for (int o = 1; o < hch; o <<= 1) ss += __shfl_xor(ss, o, 64);
      const float rs = 1.f / sqrtf(ss / (float)hd + eps);
      const uint16_t *gain = h < nq ? gq : gk;
      const u32x4_t ga = ld_u32x4(gain + t0), gb = ld_u32x4(gain + t0 + half);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        fa[2 * e] = fa[2 * e] * rs * bf16_lo(ga[e]);
        fa[2 * e + 1] = fa[2 * e + 1] * rs * bf16_hi(ga[e]);
        fb[2 * e] = fb[2 * e] * rs * bf16_lo(gb[e]);
        fb[2 * e + 1] = fb[2 * e + 1] * rs * bf16_hi(gb[e]);
      }
    }
    u32x4_t ra, rb;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float c0 = cs[t0 + 2 * e], s0 = sn[t0 + 2 * e], c1 = cs[t0 + 2 * e + 1], s1 = sn[t0 + 2 * e + 1];
      const float a0 = fa[2 * e], a1 = fa[2 * e + 1], b0 = fb[2 * e], b1 = fb[2 * e + 1];
      ra[e] = pack_bf16x2(a0 * c0 - b0 * s0, a1 * c1 - b1 * s1);
      rb[e] = pack_bf16x2(a0 * s0 + b0 * c0, a1 * s1 + b1 * c1);
    }
    if (h < nq) {
      st_u32x4(row + h * hd + t0, ra);
      st_u32x4(row + h * hd + t0 + half, rb);
    } else if (page_ok) {
      const size_t e0 = (((size_t)page * nkv + (h - nq)) * kPageSize + slot) * hd;
      if constexpr (F8) {
        uint8_t *dst = reinterpret_cast<uint8_t *>(kc) + e0;
        *reinterpret_cast<u32x2_t *>(dst + t0) = e4m3x8_of_bf16x8(ra, ks);
        *reinterpret_cast<u32x2_t *>(dst + t0 + half) = e4m3x8_of_bf16x8(rb, ks);
      } else {
        st_u32x4(kc + e0 + t0, ra);
        st_u32x4(kc + e0 + t0 + half, rb);
      }
    }
  }
  // v: plain copy, 16 bytes per thread
  const int v_lo = max(h_lo, nq + nkv) - (nq + nkv), v_hi = h_hi - (nq + nkv);
  if (page_ok && v_lo < v_hi) {
    const uint16_t *vsrc = row + (nq + nkv + v_lo) * hd;
    const int vch = (v_hi - v_lo) * hd / 8;
    for (int i = threadIdx.x; i < vch; i += blockDim.x) {
      const int kh = v_lo + (i * 8) / hd, dd = (i * 8) % hd;
      const size_t e0 = (((size_t)page * nkv + kh) * kPageSize + slot) * hd + dd;
      if constexpr (F8)
        *reinterpret_cast<u32x2_t *>(reinterpret_cast<uint8_t *>(vc) + e0) = e4m3x8_of_bf16x8(ld_u32x4(vsrc + i * 8), vs);
      else
        st_u32x4(vc + e0, ld_u32x4(vsrc + i * 8));
    }
  }
}

hipError_t launch_qkv_rope_append(const Shape &s, const float *part, int splits, const float *ssq, uint16_t *qkv,
                                  const KV &kv, const DevMeta &m, hipStream_t st, const uint16_t *gq,
                                  const uint16_t *gk) {
  if (m.T <= 0) return hipSuccess;
  if (s.qkn && (!gq || !gk)) return hipErrorInvalidValue;
  if (s.qkv_cols() % 4) return hipErrorInvalidValue;
  const QkvPartials qp{part, ssq, splits, s.hidden, s.eps};
  // four heads per block: a row's split-K sum is spread over several CUs
  const int groups = (s.nq + 2 * s.nkv + 3) / 4;
#define EB_ROPE_APPEND(F8_, QKN_)                                                                                   \
  hipLaunchKernelGGL((k_rope_append<F8_, QKN_, true>), dim3(m.T, groups), dim3(256), 0, st, qkv, kv.k, kv.v, kv.bt, \
                     kv.num_pages, kv.max_pages, m, s.nq, s.nkv, s.hd, log2((double)s.theta), kv.ks, kv.vs, gq, gk, \
                     s.eps, qp)
  if (kv.f8) {
    if (s.qkn)
      EB_ROPE_APPEND(true, true);
    else
      EB_ROPE_APPEND(true, false);
  } else {
    if (s.qkn)
      EB_ROPE_APPEND(false, true);
    else
      EB_ROPE_APPEND(false, false);
  }
#undef EB_ROPE_APPEND
  return hipGetLastError();
}

hipError_t launch_rope_append(const Shape &s, uint16_t *qkv, const KV &kv, const DevMeta &m, hipStream_t st,
                              const uint16_t *gq, const uint16_t *gk) {
  if (m.T <= 0) return hipSuccess;
  if (s.qkn && (!gq || !gk)) return hipErrorInvalidValue;
#define EB_ROPE_APPEND(F8_, QKN_)                                                                                   \
  hipLaunchKernelGGL((k_rope_append<F8_, QKN_>), dim3(m.T), dim3(256), 0, st, qkv, kv.k, kv.v, kv.bt, kv.num_pages, \
                     kv.max_pages, m, s.nq, s.nkv, s.hd, log2((double)s.theta), kv.ks, kv.vs, gq, gk, s.eps)
  if (kv.f8) {
    if (s.qkn)
      EB_ROPE_APPEND(true, true);
    else
      EB_ROPE_APPEND(true, false);
  } else {
    if (s.qkn)
      EB_ROPE_APPEND(false, true);
    else
      EB_ROPE_APPEND(false, false);
  }
#undef EB_ROPE_APPEND
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Dense gather of cached positions through the block tables (bit-exact
// paging probe).  One thread per (position, kv head, 16-byte chunk); ES
// bytes per element (2: bf16, 1: 8-bit codes, copied as they are).
// ---------------------------------------------------------------------------
template <int ES>
__global__ __launch_bounds__(256) void k_gather_kv(const uint8_t *__restrict__ kc, const uint8_t *__restrict__ vc,
                                                   const int32_t *__restrict__ bt, int num_pages, int max_pages,
                                                   DevMeta m, int nkv, int hd, uint8_t *__restrict__ ok,
                                                   uint8_t *__restrict__ ov) {
  const int chunks = hd * ES / 16;
  const long total = (long)m.gather_off[m.S] * nkv * chunks;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += (long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % chunks);
    const long pk = idx / chunks;
    const int kh = (int)(pk % nkv);
    const int gp = (int)(pk / nkv);
    int lo = 0, hi = m.S - 1;
    while (lo < hi) {  // last request whose gather offset is <= gp
      const int mid = (lo + hi + 1) >> 1;
      if (m.gather_off[mid] <= gp) lo = mid; else hi = mid - 1;
    }
    const int seq = lo;
    const int p = gp - m.gather_off[seq];
    const int page = bt[(size_t)seq * max_pages + p / kPageSize];
    u32x4_t kv4 = {0, 0, 0, 0}, vv4 = {0, 0, 0, 0};
    if (page >= 0 && page < num_pages) {
      const size_t src = ((((size_t)page * nkv + kh) * kPageSize + p % kPageSize) * hd) * ES + c * 16;
      kv4 = ld_u32x4(kc + src);
      vv4 = ld_u32x4(vc + src);
    }
    const size_t dst = (((size_t)gp * nkv + kh) * hd) * ES + c * 16;
    st_u32x4(ok + dst, kv4);
    st_u32x4(ov + dst, vv4);
  }
}

hipError_t launch_gather_kv(const Shape &s, const KV &kv, const DevMeta &m, uint16_t *out_k, uint16_t *out_v,
                            hipStream_t st) {
  if (m.S <= 0) return hipSuccess;
  uint8_t *ok = reinterpret_cast<uint8_t *>(out_k), *ov = reinterpret_cast<uint8_t *>(out_v);
  if (kv.f8)
    hipLaunchKernelGGL(k_gather_kv<1>, dim3(1024), dim3(256), 0, st, kv.k8(), kv.v8(), kv.bt, kv.num_pages,
                       kv.max_pages, m, s.nkv, s.hd, ok, ov);
  else
    hipLaunchKernelGGL(k_gather_kv<2>, dim3(1024), dim3(256), 0, st, reinterpret_cast<const uint8_t *>(kv.k),
                       reinterpret_cast<const uint8_t *>(kv.v), kv.bt, kv.num_pages, kv.max_pages, m, s.nkv, s.hd,
                       ok, ov);
  return hipGetLastError();
}

}  // namespace eb
