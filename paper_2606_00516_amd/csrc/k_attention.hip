// Paged attention for one step: split-K decode attention with a log-sum-exp
// combine, LDS-tiled causal prefill attention on bf16 MFMA, and a mixed
// launch that runs both kinds of work items in one grid.
//
// Cache layout: [page][kv head][16 slots][head_dim] bf16, so one (page, kv
// head) block is 16 * head_dim * 2 bytes, contiguous.  Query head h reads kv
// head h / G; a work item owns one kv head and serves all G of its query
// heads, so each cached byte is read once per item.
#include <math.h>

#include <type_traits>

#include "device_common.h"
#include "eb_internal.h"

namespace eb {

constexpr float kNegInf = -__builtin_inff();

// Cache words a lane holds for 8 consecutive dims of one token: 16 bytes of
// bf16, or 8 bytes of 8-bit codes (F8), turned into bf16 words when used
// (the codes' values are exact in bf16; the scales enter the score scale and
// the output normalisation).
template <bool F8>
using RawT = typename std::conditional<F8, u32x2_t, u32x4_t>::type;
template <bool F8>
EB_DEV u32x4_t raw_bf16(const RawT<F8> &w) {
  if constexpr (F8)
    return e4m3x8_to_bf16x8(w);
  else
    return w;
}

// ===========================================================================
// Decode: one work unit = (decode request, split of 32 pages, kv head) with
// NW wavefronts streaming pages w, w+NW, .. of the split, or, for a request
// with at most 64 keys, (decode request, 4 kv heads) with one wavefront per
// kv head.  Lane layout
// over a 16 x HD page block: each 16-byte load instruction covers 1 KiB, lane
// l holding 8 dims of one token; LPT = HD/8 lanes share a token.  Scores are
// reduced over those lanes with DPP; each lane keeps its own running
// (max, sum, output) over the tokens it sees, and the partial states are
// merged at the end (shuffles within the wave, LDS across waves).
// ===========================================================================
template <int HD, int G, int NW>
struct DecodeTraits {
  static constexpr int LPT = HD / 8;   // lanes per token
  static constexpr int TG = 64 / LPT;  // tokens per load instruction
  static constexpr int NLD = HD / 32;  // load instructions per page block = tokens per lane per page
  static constexpr int LDS_BYTES = NW * G * (HD + 2) * 4;
};

// Merge running softmax state (m, l, o) with another one.
template <int N>
__device__ __forceinline__ void lse_merge(float &m, float &l, float *o, float m2, float l2, const float *o2) {
  const float mx = fmaxf(m, m2);
  const float a = (m == kNegInf) ? 0.f : fast_exp2(m - mx);
  const float b = (m2 == kNegInf) ? 0.f : fast_exp2(m2 - mx);
  l = l * a + l2 * b;
#pragma unroll
  for (int i = 0; i < N; ++i) o[i] = o[i] * a + o2[i] * b;
  m = mx;
}

// Page buffers a wavefront keeps in flight while it works on another page
// (three named register sets, rotated by hand so they stay in registers).
template <int HD, int NLD, bool F8>
__device__ __forceinline__ void decode_load_page(RawT<F8> (&k)[NLD], RawT<F8> (&v)[NLD], const KV kv,
                                                 const int32_t *bt, int p, int pg1, int nkv, int kh, int lane) {
  // page p of the split is wave-uniform; past the end (or a bad table
  // entry) the descriptors cover zero bytes and the loads return zero
  const int phys = p < pg1 ? bt[p] : -1;
  const bool ok = phys >= 0 && phys < kv.num_pages;
  const size_t off = ok ? ((size_t)phys * nkv + kh) * kPageSize * HD : 0;
  if constexpr (F8) {
    // a lane's 8 codes sit at byte 8 lane + 512 j of the block (same tokens
    // and dims as the 16 bf16 bytes below)
    const int bytes8 = __builtin_amdgcn_readfirstlane(ok ? kPageSize * HD : 0);
    const buf_rsrc_t rk = make_rsrc(kv.k8() + off, bytes8);
    const buf_rsrc_t rv = make_rsrc(kv.v8() + off, bytes8);
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      k[j] = buf_ld_u32x2<kAuxNT>(rk, lane * 8 + j * 512);
      v[j] = buf_ld_u32x2<kAuxNT>(rv, lane * 8 + j * 512);
    }
  } else {
    const int bytes = ok ? kPageSize * HD * 2 : 0;
    const buf_rsrc_t rk = make_rsrc(kv.k + off, bytes);
    const buf_rsrc_t rv = make_rsrc(kv.v + off, bytes);
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      k[j] = buf_ld_u32x4<kAuxNT>(rk, lane * 16 + j * 1024);
      v[j] = buf_ld_u32x4<kAuxNT>(rv, lane * 16 + j * 1024);
    }
  }
}

// Online-softmax update of one lane's (max, sum, output) state with the
// tokens of one page it holds.
template <int HD, int G, bool F8>
__device__ __forceinline__ void decode_page_update(const RawT<F8> (&kr)[HD / 32], const RawT<F8> (&vr)[HD / 32],
                                                   const u32x4_t (&qw)[G], float (&mrun)[G], float (&lrun)[G],
                                                   float (&o)[G][8], int p, int k1, int lane, float qscale) {
  constexpr int LPT = HD / 8, TG = 64 / LPT, NLD = HD / 32;
  u32x4_t k[NLD], v[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) {
    k[j] = raw_bf16<F8>(kr[j]);
    v[j] = raw_bf16<F8>(vr[j]);
  }
  bool valid[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j) valid[j] = p * kPageSize + j * TG + lane / LPT < k1;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float sc[NLD];
    float mx = mrun[h];
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc = dot2_bf16(qw[h][i], k[j][i], acc);
      acc = group_sum<LPT>(acc) * qscale;
      sc[j] = valid[j] ? acc : kNegInf;
      mx = fmaxf(mx, sc[j]);
    }
    const float alpha = (mrun[h] == kNegInf) ? 0.f : fast_exp2(mrun[h] - mx);
    float l = lrun[h] * alpha;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[h][i] *= alpha;
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      // masked tokens: probability 0, value never read (may be NaN poison)
      const float pj = valid[j] ? fast_exp2(sc[j] - mx) : 0.f;
      l += pj;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t w = valid[j] ? v[j][i] : 0u;
        o[h][2 * i] = fmaf(pj, bf16_lo(w), o[h][2 * i]);
        o[h][2 * i + 1] = fmaf(pj, bf16_hi(w), o[h][2 * i + 1]);
      }
    }
    lrun[h] = l;
    mrun[h] = mx;
  }
}

// Stream pages p_first, p_first + stride, .. (< pg1) of one (request, kv
// head) through a ring of page buffers (three for G <= 2, two for larger
// groups, whose accumulators need the registers), rotated in straight-line
// code; pages past the end load as zeros without memory traffic and are
// masked out.  Scheduling barriers keep page loads and page updates in
// program order, so the wait before an update covers only that page.
template <int HD, int G, bool F8>
__device__ __forceinline__ void decode_stream(const KV kv, const int32_t *bt, int p_first, int stride, int pg1, int k1,
                                              int nkv, int kh, int lane, float qscale, const u32x4_t (&qw)[G],
                                              float (&mrun)[G], float (&lrun)[G], float (&o)[G][8]) {
  constexpr int NLD = HD / 32;
  RawT<F8> ka[NLD], va[NLD], kb[NLD], vb[NLD], kc[NLD], vc[NLD];
#define EB_LOAD(K_, V_, P_)                                                  \
  decode_load_page<HD, NLD, F8>(K_, V_, kv, bt, P_, pg1, nkv, kh, lane);     \
  __builtin_amdgcn_sched_barrier(0);
#define EB_UPDATE(K_, V_, P_)                                                    \
  decode_page_update<HD, G, F8>(K_, V_, qw, mrun, lrun, o, P_, k1, lane, qscale); \
  __builtin_amdgcn_sched_barrier(0);
  EB_LOAD(ka, va, p_first)
  EB_LOAD(kb, vb, p_first + stride)
  if constexpr (G <= 2) {
    EB_LOAD(kc, vc, p_first + 2 * stride)
    for (int p = p_first; p < pg1; p += 3 * stride) {
      EB_UPDATE(ka, va, p)
      EB_LOAD(ka, va, p + 3 * stride)
      EB_UPDATE(kb, vb, p + stride)
      EB_LOAD(kb, vb, p + 4 * stride)
      EB_UPDATE(kc, vc, p + 2 * stride)
      EB_LOAD(kc, vc, p + 5 * stride)
    }
  } else {
    (void)kc;
    (void)vc;
    for (int p = p_first; p < pg1; p += 2 * stride) {
      EB_UPDATE(ka, va, p)
      EB_LOAD(ka, va, p + 2 * stride)
      EB_UPDATE(kb, vb, p + stride)
      EB_LOAD(kb, vb, p + 3 * stride)
    }
  }
#undef EB_LOAD
#undef EB_UPDATE
}

// Merge the token groups of a wave (lanes with equal lane % LPT): afterwards
// every lane holds the wave's state for its 8 dims.
template <int HD, int G>
__device__ __forceinline__ void decode_merge_lanes(float (&mrun)[G], float (&lrun)[G], float (&o)[G][8]) {
  constexpr int LPT = HD / 8;
#pragma unroll
  for (int mask = LPT; mask < 64; mask <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float o2[8];
      const float m2 = shfl_xor_f32(mrun[h], mask);
      const float l2 = shfl_xor_f32(lrun[h], mask);
#pragma unroll
      for (int i = 0; i < 8; ++i) o2[i] = shfl_xor_f32(o[h][i], mask);
      lse_merge<8>(mrun[h], lrun[h], o[h], m2, l2, o2);
    }
  }
}

// Merge the per-wave softmax states a work unit left in LDS ([wave][h][HD]
// outputs, then [wave][h][2] max and sum) and write the unit's result: the
// final row (one split) or a partial for the combine.
// vscale: the value scale of an 8-bit cache (1 for bf16: exact).
// The decode request and work of a unit.  Units come in three runs (the
// plan's launch order): the full 32-page splits, request by request (each
// wavefront finds the request by a 64-way search over the records' first
// full-split units: lane i probes the i-th of 64 evenly spaced records, the
// ballot keeps the last one at or below the unit; one round of loads for 64
// requests, two for 4096); then the shorter last splits of the requests
// listed longest first, n_kv units each; then the requests of at most
// kShortDecodeKeys keys.  Every unit computes the same result wherever it
// sits in the order.
struct DecUnit {
  int local;      // split * n_kv + kv head, or the head group of a short request
  int split_off;  // first global split index of the request
  int nsplit;     // splits of the request
  int seq, row, nkeys;
};

__device__ __forceinline__ DecUnit find_decode_unit(const DevMeta &md, int unit, int nkv) {
  int d, local;
  if (unit < md.n_full_units) {
    const int lane = threadIdx.x & 63;
    int lo = 0, n = md.n_dec;  // the request lies in [lo, lo + n)
    while (n > 1) {
      const int step = (n + 63) >> 6;
      const int idx = lo + lane * step;
      // first full-split units do not decrease with the request index, so
      // the probes at or below the unit are a prefix of the lanes
      const bool ok = idx < lo + n && md.dec_info[(size_t)idx * kDecInfoInts] <= unit;
      const int last = __builtin_popcountll(__builtin_amdgcn_ballot_w64(ok)) - 1;
      const int nlo = lo + last * step;
      n = min(step, lo + n - nlo);
      lo = nlo;
    }
    d = __builtin_amdgcn_readfirstlane(lo);
    local = unit - md.dec_info[(size_t)d * kDecInfoInts];
  } else if (unit < md.n_full_units + md.n_part * nkv) {
    const int u = unit - md.n_full_units;
    const int i = u / nkv;
    d = md.dec_part[i];
    local = (md.dec_info[(size_t)d * kDecInfoInts + 5] - 1) * nkv + (u - i * nkv);  // the last split
  } else {
    const int nsu = (nkv + kShortDecodeHeads - 1) / kShortDecodeHeads;
    const int u = unit - md.n_full_units - md.n_part * nkv;
    const int i = u / nsu;
    d = md.dec_short[i];
    local = u - i * nsu;
  }
  const int32_t *r = md.dec_info + (size_t)d * kDecInfoInts;
  DecUnit du;
  du.local = local;
  du.split_off = r[1];
  du.seq = r[2];
  du.row = r[3];
  du.nkeys = r[4];
  du.nsplit = r[5];
  return du;
}

template <int HD, int G, int NW>
__device__ __forceinline__ void decode_merge_waves(const float *lo_, const float *lml, int row, int kh, int nq,
                                                   int nkv, int item, int nsplit, uint16_t *__restrict__ out,
                                                   float *__restrict__ part_o, float *__restrict__ part_ml,
                                                   float vscale) {
  __syncthreads();
  for (int e = threadIdx.x; e < G * HD; e += blockDim.x) {
    const int h = e / HD, dim = e - h * HD;
    float mx = kNegInf;
#pragma unroll
    for (int w = 0; w < NW; ++w) mx = fmaxf(mx, lml[(w * G + h) * 2]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = lml[(w * G + h) * 2];
      const float a = (mw == kNegInf) ? 0.f : fast_exp2(mw - mx);
      L += a * lml[(w * G + h) * 2 + 1];
      O += a * lo_[(w * G + h) * HD + dim];
    }
    O *= vscale;
    const int qh = kh * G + h;
    if (nsplit == 1) {
      out[(size_t)row * nq * HD + qh * HD + dim] = (uint16_t)f32_to_bf16_bits(O / L);
    } else {
      const size_t slot = ((size_t)item * nkv + kh) * G + h;
      part_o[slot * HD + dim] = O;
      if (dim == 0) {
        part_ml[slot * 2] = mx;
        part_ml[slot * 2 + 1] = L;
      }
    }
  }
  __syncthreads();
}

template <int HD, int G>
__device__ __forceinline__ void decode_load_q(const uint16_t *__restrict__ qkv, int cols, int row, int kh, int lane,
                                              u32x4_t (&qw)[G], float (&mrun)[G], float (&lrun)[G],
                                              float (&o)[G][8]) {
  const int dq = (lane % (HD / 8)) * 8;
#pragma unroll
  for (int h = 0; h < G; ++h) qw[h] = ld_u32x4(qkv + (size_t)row * cols + (kh * G + h) * HD + dq);
#pragma unroll
  for (int h = 0; h < G; ++h) {
    mrun[h] = kNegInf;
    lrun[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[h][i] = 0.f;
  }
}

// ---------------------------------------------------------------------------
// Decode on the matrix cores, used for the larger query groups (G >= 4),
// where the per-lane form above spends most of its issue slots on redundant
// score reductions and exponentials.  Per wavefront and pair of pages (A, B)
// of one kv head:
//   S^T[token][head] = K Q^T     A = K in its cache layout (lane l: token
//                                l % 16, dims 8 (l / 16) + 32 ks ..), B = Q^T
//   V pieces         = V Sel_h   Sel_h is the 0/1 matrix that keeps dims
//                                16 h .. 16 h + 15 of a 32-dim chunk, so the
//                                product is exact and leaves lane l with 4
//                                consecutive tokens of one dim
//   O^T[dim][head]  += V^T P^T   keys ordered (A tokens 4 (l/16) .. + 3, B
//                                tokens 4 (l/16) .. + 3) in both operands
// The 16 MFMA columns are query heads (G of them used): lane l serves head
// l % 16 and holds 4 tokens of each page's scores, so only the running max
// crosses lanes (two steps).  P enters the product rounded to bf16; the sum
// l is kept in fp32.
// ---------------------------------------------------------------------------
template <int G>
constexpr bool kDecodeMfma = G >= 4;

// Page blocks reach LDS by direct loads (no registers): each 16-byte chunk
// of a block goes to a position swizzled by its token, so that every load
// instruction still covers whole 256-byte token rows of HBM and the MFMA
// operand reads (16 tokens x one chunk per quarter-wave) hit 16 different
// bank groups.  A wavefront owns four page slots (K block then V block)
// and keeps three pages in flight while it works on the fourth.
template <int HD, bool F8 = false>
struct MdecTraits {
  static constexpr int ES = F8 ? 1 : 2;            // bytes per cached element
  static constexpr int BLK = kPageSize * HD * ES;  // bytes of one (page, kv head) block
  static constexpr int SLOT = 2 * BLK;             // K block, then V block
  static constexpr int NDMA = BLK / 1024;          // 1 KiB load instructions per block
  static constexpr int ROW = HD * ES;              // bytes per token row
  static_assert(NDMA >= 1, "block of at least 1 KiB");
};

// 16-byte chunk position exchange of token row t: rows of 256 bytes (bf16,
// HD 128) take t & 15, 128-byte rows t & 7, 64-byte rows (t >> 1) & 3 ...
template <int HD, bool F8 = false>
EB_DEV int mdec_swz(int t) {
  constexpr int ROW = MdecTraits<HD, F8>::ROW;
  return ROW == 256 ? (t & 15) : ROW == 128 ? ((F8 ? t : (t >> 1)) & 7) : ((t >> 1) & 3);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Start the loads of page p (physical page phys, -1 past the end) K and V
// blocks into a slot; slots at or past k1 (and pages past the end or with a
// bad table entry) land as zeros without memory traffic, so cache poison
// never reaches the products.
template <int HD, bool F8>
__device__ __forceinline__ void mdec_dma_page(uint8_t *slot, const uint32_t *goff, const KV kv, int phys, int p,
                                              int k1, int nkv, int kh) {
  using Tr = MdecTraits<HD, F8>;
  const int nvalid = min(max(k1 - p * kPageSize, 0), kPageSize);
  const bool ok = phys >= 0 && phys < kv.num_pages;
  const size_t off = ok ? ((size_t)phys * nkv + kh) * kPageSize * HD : 0;
  // wave-uniform by construction; said so, so the descriptor stays scalar
  const int bytes = __builtin_amdgcn_readfirstlane(ok ? nvalid * Tr::ROW : 0);
  const buf_rsrc_t rk = F8 ? make_rsrc(kv.k8() + off, bytes) : make_rsrc(kv.k + off, bytes);
  const buf_rsrc_t rv = F8 ? make_rsrc(kv.v8() + off, bytes) : make_rsrc(kv.v + off, bytes);
#pragma unroll
  for (int i = 0; i < Tr::NDMA; ++i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void_t *)(slot + i * 1024), 16, goff[i], 0, 0, kAuxNT);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void_t *)(slot + Tr::BLK + i * 1024), 16, goff[i], 0, 0,
                                             kAuxNT);
  }
}

// Upper halves of two fp32 values that hold bf16 numbers exactly, packed.
EB_DEV uint32_t bf16_pair_exact(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}


// Online-softmax update with the page in a slot; the page holds at least one
// key below k1, so the new running max is finite.
template <int HD, bool F8>
__device__ __forceinline__ void mdec_page_update(const uint8_t *slot, const u32x4_t (&qb)[HD / 32],
                                                 const u32x4_t (&sel)[2], float &mrun, float &lsum,
                                                 f32x4_t (&oacc)[HD / 16], int p, int k1, int lane, float qscale) {
  using Tr = MdecTraits<HD, F8>;
  constexpr int NKS = HD / 32;
  const int r = lane & 15, g = lane >> 4;
  const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
  const uint8_t *rowp = slot + r * Tr::ROW;
  const int sw = mdec_swz<HD, F8>(r);
  // dims 8 g + 32 ks .. + 7 of token r: a 16-byte chunk of bf16, or half of
  // one of 8-bit codes
  auto dims8 = [&](const uint8_t *base, int ks) -> u32x4_t {
    if constexpr (F8)
      return e4m3x8_to_bf16x8(
          *reinterpret_cast<const u32x2_t *>(base + ((((g >> 1) + 2 * ks) ^ sw) << 4) + ((g & 1) << 3)));
    else
      return *reinterpret_cast<const u32x4_t *>(base + (((g + 4 * ks) ^ sw) << 4));
  };
  f32x4_t sa = zero;
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) sa = mfma16x16x32(dims8(rowp, ks), qb[ks], sa);
  float s[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) s[j] = sa[j] * qscale;
  if (p * kPageSize + kPageSize > k1) {  // wave-uniform: the page reaches past the last key
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (p * kPageSize + 4 * g + j >= k1) s[j] = kNegInf;
  }
  float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
  mx = fmaxf(mx, shfl_xor_f32(mx, 16));
  mx = fmaxf(mx, shfl_xor_f32(mx, 32));
  const float mnew = fmaxf(mrun, mx);
  const float alpha = (mrun == kNegInf) ? 0.f : fast_exp2(mrun - mnew);
  float pr[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) pr[j] = fast_exp2(s[j] - mnew);
  lsum = lsum * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
  mrun = mnew;
  // P^T (keys 4 g .. 4 g + 3 of this lane's head) as the B operand of the
  // 16x16x16 product
  const u32x2_t pt = {bf16_pair_rne(pr[0], pr[1]), bf16_pair_rne(pr[2], pr[3])};
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const u32x4_t vv = dims8(rowp + Tr::BLK, ks);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4_t t = mfma16x16x32(vv, sel[h], zero);  // V[4 g + j][32 ks + 16 h + r]
      const u32x2_t a = {bf16_pair_exact(t[0], t[1]), bf16_pair_exact(t[2], t[3])};
      oacc[2 * ks + h] = mfma16x16x16(a, pt, oacc[2 * ks + h] * alpha);
    }
  }
}

// Stream pages p_first, p_first + stride, .. (< pg1) through the wave's
// NSLOT slots (NSLOT - 1 pages in flight while one is consumed).  Lane l of
// vbt holds the physical page of page pbase + l (all pages streamed lie in
// pbase .. pbase + 63), so no page waits for a table load.  Loads of pages
// past the end cost no memory traffic; every load has landed when this
// returns.
template <int HD, int NSLOT, bool F8>
__device__ __forceinline__ void mdec_stream(uint8_t *s0, uint8_t *s1, uint8_t *s2, uint8_t *s3, const KV kv,
                                            int vbt, int pbase, int p_first, int stride, int pg1, int k1, int nkv,
                                            int kh, int lane, float qscale, const u32x4_t (&qb)[HD / 32],
                                            const u32x4_t (&sel)[2], float &mrun, float &lsum,
                                            f32x4_t (&oacc)[HD / 16]) {
  using Tr = MdecTraits<HD, F8>;
  static_assert(NSLOT >= 2 && NSLOT <= 4, "ring depth");
  static_assert(kDecodePagesPerSplit <= 64 && (kShortDecodeKeys + kPageSize - 1) / kPageSize <= 64,
                "a wave's pages fit one table entry per lane");
  uint32_t goff[Tr::NDMA];
#pragma unroll
  for (int i = 0; i < Tr::NDMA; ++i) {
    const int e = i * 1024 + lane * 16;  // byte of the slot block this lane fills
    const int t = e / Tr::ROW, u = (e % Tr::ROW) >> 4;
    goff[i] = (uint32_t)(t * Tr::ROW + ((u ^ mdec_swz<HD, F8>(t)) << 4));
  }
#define EB_DMA(S_, P_)                                                                             \
  mdec_dma_page<HD, F8>(S_, goff, kv, (P_) < pg1 ? __builtin_amdgcn_readlane(vbt, (P_) - pbase) : -1, P_, k1, \
                        nkv, kh);                                                                    \
  __builtin_amdgcn_sched_barrier(0);
#define EB_UPD(S_, P_)                                                                  \
  if ((P_) < pg1) mdec_page_update<HD, F8>(S_, qb, sel, mrun, lsum, oacc, P_, k1, lane, qscale); \
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (NSLOT == 2) {
    (void)s2;
    (void)s3;
    EB_DMA(s0, p_first)
    for (int p = p_first; p < pg1; p += 2 * stride) {
      EB_DMA(s1, p + stride)
      EB_UPD(s0, p)
      EB_DMA(s0, p + 2 * stride)
      EB_UPD(s1, p + stride)
    }
  } else if constexpr (NSLOT == 3) {
    (void)s3;
    EB_DMA(s0, p_first)
    EB_DMA(s1, p_first + stride)
    for (int p = p_first; p < pg1; p += 3 * stride) {
      EB_DMA(s2, p + 2 * stride)
      EB_UPD(s0, p)
      EB_DMA(s0, p + 3 * stride)
      EB_UPD(s1, p + stride)
      EB_DMA(s1, p + 4 * stride)
      EB_UPD(s2, p + 2 * stride)
    }
  } else {
    EB_DMA(s0, p_first)
    EB_DMA(s1, p_first + stride)
    EB_DMA(s2, p_first + 2 * stride)
    for (int p = p_first; p < pg1; p += 4 * stride) {
      EB_DMA(s3, p + 3 * stride)
      EB_UPD(s0, p)
      EB_DMA(s0, p + 4 * stride)
      EB_UPD(s1, p + stride)
      EB_DMA(s1, p + 5 * stride)
      EB_UPD(s2, p + 2 * stride)
      EB_DMA(s2, p + 6 * stride)
      EB_UPD(s3, p + 3 * stride)
    }
  }
#undef EB_DMA
#undef EB_UPD
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// q of the G heads of kv head kh as the B operand (columns >= G zero), the
// two selection matrices, and the empty softmax state.
template <int HD, int G>
__device__ __forceinline__ void mdec_init(const uint16_t *__restrict__ qkv, int cols, int row, int kh, int lane,
                                          u32x4_t (&qb)[HD / 32], u32x4_t (&sel)[2], float &mrun, float &lsum,
                                          f32x4_t (&oacc)[HD / 16]) {
  const int c = lane & 15, g = lane >> 4;
  const bool live = c < G;
  const uint16_t *src = qkv + (size_t)row * cols + (kh * G + (live ? c : 0)) * HD + g * 8;
#pragma unroll
  for (int ks = 0; ks < HD / 32; ++ks) {
    const u32x4_t v = ld_u32x4(src + ks * 32);
    qb[ks] = live ? v : u32x4_t{0u, 0u, 0u, 0u};
  }
  // Sel_h[k][c] = 1 where k = c + 16 h: lane (c, g) holds k = 8 g .. 8 g + 7
  const uint32_t one = (c & 1) ? 0x3F800000u : 0x3F80u;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const bool hit = g == 2 * h + (c >> 3);
#pragma unroll
    for (int e = 0; e < 4; ++e) sel[h][e] = (hit && e == ((c & 7) >> 1)) ? one : 0u;
  }
  mrun = kNegInf;
  lsum = 0.f;
#pragma unroll
  for (int ob = 0; ob < HD / 16; ++ob) oacc[ob] = f32x4_t{0.f, 0.f, 0.f, 0.f};
}

// One decode work unit on the matrix cores (same units as decode_item),
// run by NW wavefronts with NSLOT-deep page rings.  l0..l3: the block's
// slot arrays (NW slots of SLOT bytes each; the first NSLOT arrays are
// used); once every wave has finished streaming, the cross-wave merge puts
// the outputs in l0 and the (max, sum) pairs in l1.
template <int HD, int G, int NW, int NSLOT, bool F8, int SLOT>
__device__ __forceinline__ void decode_item_mfma(const uint16_t *__restrict__ qkv, int nq, int nkv, const KV kv,
                                                 const DevMeta md, int unit, uint16_t *__restrict__ out,
                                                 float *__restrict__ part_o, float *__restrict__ part_ml, uint8_t *l0,
                                                 uint8_t *l1, uint8_t *l2, uint8_t *l3) {
  constexpr int SPLIT = kDecodePagesPerSplit * kPageSize;
  constexpr int NOB = HD / 16;
  static_assert(SLOT >= MdecTraits<HD, F8>::SLOT, "slot holds a page's K and V blocks");
  static_assert(NW * G * HD * 4 <= NW * SLOT && NW * G * 2 * 4 <= NW * SLOT, "merge area");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cols = (nq + 2 * nkv) * HD;
  const float qscale = F8 ? kLog2e / sqrtf((float)HD) * kv.ks : kLog2e / sqrtf((float)HD);
  const float vscale = F8 ? kv.vs : 1.f;
  const int c = lane & 15, g = lane >> 4;
  uint8_t *w0 = l0 + wave * SLOT, *w1 = l1 + wave * SLOT, *w2 = l2 + wave * SLOT, *w3 = l3 + wave * SLOT;

  const DecUnit du = find_decode_unit(md, unit, nkv);
  const int local = du.local, nkeys = du.nkeys, row = du.row;
  const int32_t *bt = kv.bt + (size_t)du.seq * kv.max_pages;
  u32x4_t qb[HD / 32], sel[2];
  float mrun, lsum;
  f32x4_t oacc[NOB];

  if (nkeys <= kShortDecodeKeys) {
    // one wavefront per kv head, all its pages, output written directly
    for (int hw = wave; hw < kShortDecodeHeads; hw += NW) {
      const int kh = local * kShortDecodeHeads + hw;
      if (kh >= nkv) break;
      const int npg = (nkeys + kPageSize - 1) / kPageSize;
      const int vbt = lane < npg ? bt[lane] : -1;
      mdec_init<HD, G>(qkv, cols, row, kh, lane, qb, sel, mrun, lsum, oacc);
      mdec_stream<HD, NSLOT, F8>(w0, w1, w2, w3, kv, vbt, 0, 0, 1, npg, nkeys, nkv, kh, lane, qscale, qb, sel, mrun,
                                 lsum, oacc);
      lsum += shfl_xor_f32(lsum, 16);
      lsum += shfl_xor_f32(lsum, 32);
      if (c < G) {
        const float inv = F8 ? vscale / lsum : 1.0f / lsum;
        uint16_t *dst = out + (size_t)row * nq * HD + (kh * G + c) * HD + g * 4;
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          const u32x2_t w = {pack_bf16x2(oacc[ob][0] * inv, oacc[ob][1] * inv),
                             pack_bf16x2(oacc[ob][2] * inv, oacc[ob][3] * inv)};
          *reinterpret_cast<u32x2_t *>(dst + ob * 16) = w;
        }
      }
    }
    return;
  }

  const int split = local / nkv, kh = local - split * nkv;
  const int item = du.split_off + split;
  const int nsplit = du.nsplit;
  const int k0 = split * SPLIT;
  const int k1 = min(nkeys, k0 + SPLIT);
  const int pg0 = k0 / kPageSize, pg1 = (k1 + kPageSize - 1) / kPageSize;
  // the split's block-table entries, one per lane, fetched once
  const int vbt = pg0 + lane < pg1 ? bt[pg0 + lane] : -1;
  mdec_init<HD, G>(qkv, cols, row, kh, lane, qb, sel, mrun, lsum, oacc);
  mdec_stream<HD, NSLOT, F8>(w0, w1, w2, w3, kv, vbt, pg0, pg0 + wave, NW, pg1, k1, nkv, kh, lane, qscale, qb, sel,
                             mrun, lsum, oacc);
  lsum += shfl_xor_f32(lsum, 16);
  lsum += shfl_xor_f32(lsum, 32);
  // across the NW waves through LDS (reusing the slots once every wave is
  // done with them): [wave][h][HD] outputs in l0, [wave][h][2] in l1
  float *merge_o = reinterpret_cast<float *>(l0), *merge_ml = reinterpret_cast<float *>(l1);
  __syncthreads();
  if (c < G) {
    float *o_ = merge_o + (wave * G + c) * HD + g * 4;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
      for (int j = 0; j < 4; ++j) o_[ob * 16 + j] = oacc[ob][j];
    if (g == 0) {
      float *ml = merge_ml + (wave * G + c) * 2;
      ml[0] = mrun;
      ml[1] = lsum;
    }
  }
  decode_merge_waves<HD, G, NW>(merge_o, merge_ml, row, kh, nq, nkv, item, nsplit, out, part_o, part_ml, vscale);
}

// One decode work unit.  Unit u of decode request d (binary search over the
// unit prefix sums): a request with at most kShortDecodeKeys keys has one
// unit per 4 kv heads, each wavefront taking one kv head and all its pages
// and writing its output directly; a longer request has one unit per
// (split of 32 pages, kv head), its NW wavefronts streaming pages w, w+NW, ..
// and merging through LDS, with the result written directly (one split) or
// as a partial for the combine.  Which kind a request gets depends only on
// its own length.
template <int HD, int G, int NW, bool F8>
__device__ __forceinline__ void decode_item(const uint16_t *__restrict__ qkv, int nq, int nkv, const KV kv,
                                            const DevMeta md, int unit, uint16_t *__restrict__ out,
                                            float *__restrict__ part_o, float *__restrict__ part_ml, float *lds) {
  using Tr = DecodeTraits<HD, G, NW>;
  constexpr int LPT = Tr::LPT;
  constexpr int SPLIT = kDecodePagesPerSplit * kPageSize;
  const int lane = threadIdx.x & 63;
  // wave index made visibly uniform, so page addressing stays scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cols = (nq + 2 * nkv) * HD;
  const float qscale = F8 ? kLog2e / sqrtf((float)HD) * kv.ks : kLog2e / sqrtf((float)HD);
  const float vscale = F8 ? kv.vs : 1.f;

  const DecUnit du = find_decode_unit(md, unit, nkv);
  const int local = du.local, nkeys = du.nkeys, row = du.row;
  const int32_t *bt = kv.bt + (size_t)du.seq * kv.max_pages;
  const int dq = (lane % LPT) * 8;
  u32x4_t qw[G];
  float mrun[G], lrun[G], o[G][8];

  if (nkeys <= kShortDecodeKeys) {
    const int kh = local * kShortDecodeHeads + wave;
    if (wave >= kShortDecodeHeads || kh >= nkv) return;
    decode_load_q<HD, G>(qkv, cols, row, kh, lane, qw, mrun, lrun, o);
    decode_stream<HD, G, F8>(kv, bt, 0, 1, (nkeys + kPageSize - 1) / kPageSize, nkeys, nkv, kh, lane, qscale, qw,
                             mrun, lrun, o);
    decode_merge_lanes<HD, G>(mrun, lrun, o);
    if (lane < LPT) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float inv = F8 ? vscale / lrun[h] : 1.0f / lrun[h];
        const u32x4_t w = {pack_bf16x2(o[h][0] * inv, o[h][1] * inv), pack_bf16x2(o[h][2] * inv, o[h][3] * inv),
                           pack_bf16x2(o[h][4] * inv, o[h][5] * inv), pack_bf16x2(o[h][6] * inv, o[h][7] * inv)};
        st_u32x4(out + (size_t)row * nq * HD + (kh * G + h) * HD + dq, w);
      }
    }
    return;
  }

  const int split = local / nkv, kh = local - split * nkv;
  const int item = du.split_off + split;   // global split index (partials)
  const int nsplit = du.nsplit;
  const int k0 = split * SPLIT;
  const int k1 = min(nkeys, k0 + SPLIT);
  const int pg0 = k0 / kPageSize, pg1 = (k1 + kPageSize - 1) / kPageSize;
  decode_load_q<HD, G>(qkv, cols, row, kh, lane, qw, mrun, lrun, o);
  decode_stream<HD, G, F8>(kv, bt, pg0 + wave, NW, pg1, k1, nkv, kh, lane, qscale, qw, mrun, lrun, o);
  decode_merge_lanes<HD, G>(mrun, lrun, o);

  // across the NW waves through LDS: [wave][h][HD] outputs, then [wave][h][2]
  float *lo_ = lds;
  float *lml = lds + NW * G * HD;
  if (lane < LPT) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
#pragma unroll
      for (int i = 0; i < 8; ++i) lo_[(wave * G + h) * HD + dq + i] = o[h][i];
      if (lane == 0) {
        lml[(wave * G + h) * 2] = mrun[h];
        lml[(wave * G + h) * 2 + 1] = lrun[h];
      }
    }
  }
  decode_merge_waves<HD, G, NW>(lds, lds + NW * G * HD, row, kh, nq, nkv, item, nsplit, out, part_o, part_ml,
                                vscale);
}

// Combine the splits of one decode request for one query head:
// o = sum_s 2^(m_s - M) o_s / sum_s 2^(m_s - M) l_s with M = max_s m_s.  Lane
// s % 64 holds split s's weight; the output dims (HD / 64 per lane) sum the
// partials eight splits at a time, their loads issued together.
template <int HD, int G>
__global__ __launch_bounds__(64) void k_decode_combine(DevMeta md, const float *__restrict__ part_o,
                                                       const float *__restrict__ part_ml, uint16_t *__restrict__ out,
                                                       int nq, int nkv) {
  constexpr int DPL = HD / 64;  // dims per lane
  const int32_t *rec = md.comb_list + (size_t)blockIdx.x * kCombInfoInts;
  const int s0 = rec[0], ns = rec[1], row = rec[2];
  const int qh = blockIdx.y;
  const int kh = qh / G, h = qh - kh * G;
  const int lane = threadIdx.x;
  const size_t stride = (size_t)nkv * G;  // slots between consecutive splits
  const size_t base = ((size_t)s0 * nkv + kh) * G + h;
  float mx = kNegInf;
  for (int s = lane; s < ns; s += 64) mx = fmaxf(mx, part_ml[(base + s * stride) * 2]);
  mx = wave_max(mx);
  float den = 0.f;
  float acc[DPL];
#pragma unroll
  for (int i = 0; i < DPL; ++i) acc[i] = 0.f;
  for (int c = 0; c < ns; c += 64) {
    const int s = c + lane;
    float wgt = 0.f;
    if (s < ns) {
      const float ms = part_ml[(base + s * stride) * 2];
      wgt = (ms == kNegInf) ? 0.f : fast_exp2(ms - mx);
      den += wgt * part_ml[(base + s * stride) * 2 + 1];
    }
    const int n = min(64, ns - c);
    for (int j = 0; j < n; j += 8) {
      float o[8][DPL];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int i = 0; i < DPL; ++i)
          o[u][i] = j + u < n ? part_o[(base + (size_t)(c + j + u) * stride) * HD + lane * DPL + i] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wgt), j + u));
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[i] += a * o[u][i];
      }
    }
  }
  den = wave_sum(den);
#pragma unroll
  for (int i = 0; i < DPL; ++i)
    out[(size_t)row * nq * HD + qh * HD + lane * DPL + i] = (uint16_t)f32_to_bf16_bits(acc[i] / den);
}

// ===========================================================================
// Prefill: one work item = (request, block of BQ query positions, kv head):
// G heads x BQ positions, cut into 16-row blocks (one head, 16 positions)
// shared out over NW wavefronts (8 in the prefill-only launch, 4 inside the
// mixed launch).  Keys and values stream through LDS in tiles of 64
// positions gathered from 4 pages; the next tile's global loads are issued
// before the current tile is consumed, and a wave holding several row blocks
// reads each K and V^T fragment once for all of them.  Scores are formed
// transposed,
// S^T = K Q^T, with the 16x16x32 bf16 MFMA, so a lane holds one query column
// and the row max needs only two cross-lane steps; P^T stays in registers as
// the B operand of O^T = V^T P^T (keys permuted consistently on both
// operands), with V^T staged in LDS.  A row's arithmetic does not depend on
// which item it sits in, so both launches give the same bits.
// ===========================================================================
// Query positions per prefill item: 128 rows (G heads x 128/G positions) in
// the prefill-only launch, 64 rows (one 16-row block per wave of the 4-wave
// block: 8 positions of two heads per block for G = 8) inside the mixed
// launch, which keeps the mixed kernel to two blocks per CU; the planner's
// prefill_bq() gives the same numbers.
template <int G, bool MIXED>
constexpr int prefill_item_positions() {
  return MIXED ? 64 / G : 128 / G;
}

// V^T in LDS: row = head dimension, 68 bf16 per row; the 8-byte group of
// keys 4 g .. 4 g + 3 of row r sits at group g ^ ((r >> 4) & 7).  LDS
// serves 128 bytes per pass over 32 banks: without the exchange the
// transposing 4-byte stores (16 row groups x 2 key pairs per pass) hit 4
// banks 8 times each; with it they spread over all 32, while the 8-byte
// operand reads (16 rows per pass, 68-wide rows put consecutive rows 8
// bytes apart modulo 128) stay conflict free.  Within the operand loop the
// exchange depends only on the 16-row block, so each read keeps a constant
// offset from one of four per-lane bases.
__device__ __forceinline__ int vt_col(int r, int key) { return 4 * ((key >> 2) ^ ((r >> 4) & 7)) + (key & 3); }

template <int HD, int G, int NW, int BQ_>
struct PrefillTraits {
  static constexpr int BQ = BQ_;                 // query positions per item
  static constexpr int RB = (G * BQ / 16) / NW;  // 16-row blocks per wavefront
  static constexpr int KT = 64;                  // keys per tile
  static constexpr int KS_STRIDE = HD + 8;       // bf16 elements per K row in LDS
  static constexpr int VT_STRIDE = KT + 4;       // bf16 elements per V^T row in LDS
  static constexpr int KS_BYTES = KT * KS_STRIDE * 2;  // K tile
  static constexpr int VT_BYTES = HD * VT_STRIDE * 2;  // V^T tile
  static constexpr int LDS_BYTES = KS_BYTES + VT_BYTES;
  static constexpr int KCH = KT * (HD / 8);      // 16-byte K chunks per tile
  static constexpr int VCH = (KT / 2) * (HD / 8);  // (key pair, 8 dims) V units per tile
  static constexpr int KPT = (KCH + NW * 64 - 1) / (NW * 64);  // per thread
  static constexpr int VPT = (VCH + NW * 64 - 1) / (NW * 64);
  static_assert(RB >= 1 && RB * NW * 16 == G * BQ, "row blocks");
  // a 16-row block holds 16 positions of one head, or 16 / BQ heads of BQ
  // positions each
  static_assert(BQ % 16 == 0 || (16 % BQ == 0 && G % (16 / BQ) == 0), "row block shape");
};

template <int HD, int G, int NW, int BQ_, bool F8>
__device__ __forceinline__ void prefill_item(const uint16_t *__restrict__ qkv, int nq, int nkv, const KV kv,
                                             const DevMeta md, int tile, int kh, uint16_t *__restrict__ out,
                                             uint16_t *Ks, uint16_t *Vt) {
  using Tr = PrefillTraits<HD, G, NW, BQ_>;
  constexpr int BQ = Tr::BQ, RB = Tr::RB, KT = Tr::KT, KSS = Tr::KS_STRIDE, VTS = Tr::VT_STRIDE;
  constexpr int KCH = Tr::KCH, VCH = Tr::VCH, KPT = Tr::KPT, VPT = Tr::VPT;
  constexpr int NKS = HD / 32;  // k-steps of the QK^T product
  constexpr int NOB = HD / 16;  // 16-dim output blocks
  constexpr int NT = NW * 64;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cols = (nq + 2 * nkv) * HD;
  const int seq = md.tile_seq[tile];
  const int qb = md.tile_qb[tile];
  const int c = md.seq_ctx[seq];
  const int n = md.seq_len[seq];
  const int row0 = md.seq_row[seq];
  const int q_lo = qb * BQ;                 // first query (chunk-relative)
  const int q_hi = min(n, q_lo + BQ);       // one past the last
  const int kend = c + q_hi;                // keys needed: 0 .. kend-1
  const int klen = c + n;                   // keys that exist
  const int32_t *bt = kv.bt + (size_t)seq * kv.max_pages;
  const int npages = (klen + kPageSize - 1) / kPageSize;
  const float qscale = F8 ? kLog2e / sqrtf((float)HD) * kv.ks : kLog2e / sqrtf((float)HD);
  const int lq = lane & 15;   // query column of this lane inside a 16-row block
  const int lg = lane >> 4;   // lane group 0..3

  // row blocks of this wave: rb = wave + NW i, each HPB heads x RPH
  // positions (RPH = min(16, BQ)); lane lq serves head hb HPB + lq / RPH at
  // position q_lo + sub RPH + lq % RPH, where hb = rb % (G / HPB), sub = rb /
  // (G / HPB).  A row's arithmetic does not depend on the block shape: the
  // products and reductions are per query column.
  constexpr int RPH = BQ < 16 ? BQ : 16, HPB = 16 / RPH, HG = G / HPB;
  int hrow[RB];
  u32x4_t qreg[RB][NKS];
  int qrel[RB];
  bool qok[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    const int rb = wave + NW * i;
    const int hb = rb % HG, sub = rb / HG;
    hrow[i] = hb * HPB + lq / RPH;
    qrel[i] = q_lo + sub * RPH + lq % RPH;
    qok[i] = qrel[i] < q_hi;
    const uint16_t *src = qkv + (size_t)(row0 + qrel[i]) * cols + (kh * G + hrow[i]) * HD + lg * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qreg[i][ks] = qok[i] ? ld_u32x4(src + ks * 32) : u32x4_t{0, 0, 0, 0};
  }
  f32x4_t oacc[RB][NOB];
  float mrun[RB], lrun[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    mrun[i] = kNegInf;
    lrun[i] = 0.f;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) oacc[i][ob] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // global -> register staging of one K/V tile (keys past c + n read as 0).
  // A tile's 64 keys sit in 4 pages; their block-table entries are loaded
  // together one tile ahead of the data loads that use them, so a tile's
  // gather costs one memory round trip, overlapped with the previous tile's
  // products.  Every load reads a valid address (position 0 of the cache for
  // an absent key) and the result is zeroed afterwards: no divergent branch.
  typedef int i32x4_t __attribute__((ext_vector_type(4)));
  constexpr int PPT = KT / kPageSize;  // pages per tile
  static_assert(PPT == 4, "tile = 4 pages");
  // the block table is read-only here: through the constant address space
  // the entries (uniform per tile) come by scalar loads into scalar
  // registers, counted apart from the vector loads of K and V
  typedef const __attribute__((address_space(4))) int32_t *bt_ptr_t;
  const bt_ptr_t btc = (bt_ptr_t)bt;
  auto bt_tile = [&](int t) -> i32x4_t {
    const int p0 = t * PPT;
    i32x4_t r = {-1, -1, -1, -1};
#pragma unroll
    for (int j = 0; j < PPT; ++j)
      if (p0 + j < npages) r[j] = btc[p0 + j];
    return r;
  };
  RawT<F8> kreg[KPT], vreg[VPT][2];
  uint32_t present = 0;  // bit i: K load i, bit KPT + 2 i + e: V load (i, e)
  // The lanes of one load instruction cover 64 / (HD / 8) consecutive keys
  // of K (or twice that of V), all in one page: the page, its validity and
  // its base address are wave-uniform (scalar registers); a lane adds only
  // its row and chunk.  An absent page reads page block 0 and is zeroed.
  static_assert(HD == 64 || HD == 128, "keys of one load within one page");
  typedef typename std::conditional<F8, const uint8_t, const uint16_t>::type elem_t;
  auto page_base = [&](elem_t *arr, const i32x4_t &btv, int j, bool &ok) -> elem_t * {
    const int phys = j == 0 ? btv[0] : j == 1 ? btv[1] : j == 2 ? btv[2] : btv[3];
    ok = phys >= 0 && phys < kv.num_pages;
    return arr + (ok ? ((size_t)phys * nkv + kh) * (kPageSize * HD) : 0);
  };
  // 8 dims of one token: 16 bytes of bf16 or 8 bytes of codes
  auto ld8 = [&](elem_t *p) -> RawT<F8> {
    if constexpr (F8)
      return *reinterpret_cast<const u32x2_t *>(p);
    else
      return ld_u32x4(p);
  };
  elem_t *const kbase = reinterpret_cast<elem_t *>(kv.k), *const vbase = reinterpret_cast<elem_t *>(kv.v);
  // the data of absent keys is zeroed when staged (zeroing right after the
  // load would wait for it)
  auto fetch = [&](int t, const i32x4_t &btv) {
    const int k0 = t * KT;
    present = 0;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int u = tid + i * NT;
      const int key = u / (HD / 8), dc = u % (HD / 8);
      const int j = __builtin_amdgcn_readfirstlane(key / kPageSize);
      bool pok;
      elem_t *pb = page_base(kbase, btv, j, pok);
      kreg[i] = ld8(pb + (key % kPageSize) * HD + dc * 8);
      present |= (u < KCH && pok && k0 + key < klen ? 1u : 0u) << i;
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      const int kpair = u / (HD / 8), dc = u % (HD / 8);
      const int j = __builtin_amdgcn_readfirstlane((2 * kpair) / kPageSize);
      bool pok;
      elem_t *pb = page_base(vbase, btv, j, pok);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = 2 * kpair + e;
        vreg[i][e] = ld8(pb + (key % kPageSize) * HD + dc * 8);
        present |= (u < VCH && pok && k0 + key < klen ? 1u : 0u) << (KPT + 2 * i + e);
      }
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int u = tid + i * NT;
      if (u < KCH)
        st_u32x4(Ks + (u / (HD / 8)) * KSS + (u % (HD / 8)) * 8,
                 (present >> i) & 1u ? raw_bf16<F8>(kreg[i]) : u32x4_t{0, 0, 0, 0});
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      if (u < VCH) {
        const int kpair = u / (HD / 8), dc = u % (HD / 8);
        // rows dc * 8 .. + 7 share one group exchange (see vt_col)
        const int col = vt_col(dc * 8, 2 * kpair);
        const bool p0 = (present >> (KPT + 2 * i)) & 1u, p1 = (present >> (KPT + 2 * i + 1)) & 1u;
        const u32x4_t v0 = raw_bf16<F8>(vreg[i][0]), v1 = raw_bf16<F8>(vreg[i][1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t a0 = p0 ? v0[j] : 0u, a1 = p1 ? v1[j] : 0u;
          *reinterpret_cast<uint32_t *>(Vt + (dc * 8 + 2 * j) * VTS + col) = (a0 & 0xFFFFu) | (a1 << 16);
          *reinterpret_cast<uint32_t *>(Vt + (dc * 8 + 2 * j + 1) * VTS + col) = (a0 >> 16) | (a1 & 0xFFFF0000u);
        }
      }
    }
  };

  const int min_qpos = c + q_lo;
  const int ntiles = (kend + KT - 1) / KT;
  i32x4_t bt_next = bt_tile(1);
  fetch(0, bt_tile(0));
  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * KT;
    stage();
    __syncthreads();
    if (t + 1 < ntiles) {  // in flight while this tile is consumed
      const i32x4_t bt_cur = bt_next;
      bt_next = bt_tile(t + 2);
      fetch(t + 1, bt_cur);
    }
    // S^T blocks of every row block (keys k0 + 16 kb + 4 lg + j, query
    // column lq): a K fragment is read from LDS once for all RB blocks
    f32x4_t sc[RB][4];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) sc[i][kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const u32x4_t a = ld_u32x4(Ks + (kb * 16 + lq) * KSS + ks * 32 + lg * 8);
#pragma unroll
        for (int i = 0; i < RB; ++i) sc[i][kb] = mfma16x16x32(a, qreg[i][ks], sc[i][kb]);
      }
    uint32_t pk[RB][4][2];
    float alpha[RB];
    bool rescale[RB];
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const bool need_mask = (k0 + KT - 1) > min_qpos || !qok[i];
      const int qpos = c + qrel[i];
      // the max is taken on the raw scores (qscale > 0 keeps the order and
      // the rounding), the scale enters the exponent through one fma
      float mraw = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (need_mask) {
            const int kp = k0 + kb * 16 + lg * 4 + j;
            if (kp > qpos || !qok[i]) sc[i][kb][j] = kNegInf;
          }
          mraw = fmaxf(mraw, sc[i][kb][j]);
        }
      mraw = fmaxf(mraw, shfl_xor_f32(mraw, 16));
      mraw = fmaxf(mraw, shfl_xor_f32(mraw, 32));
      const float mx = fmaxf(mrun[i], mraw * qscale);
      alpha[i] = (mrun[i] == kNegInf) ? 0.f : fast_exp2(mrun[i] - mx);
      // masked scores are -inf, so exp2 gives 0 without a select; a row with
      // nothing visible yet keeps an offset of 0
      const float neg = mx != kNegInf ? -mx : 0.f;
      float l = lrun[i] * alpha[i];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        float p4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          p4[j] = fast_exp2(fmaf(sc[i][kb][j], qscale, neg));
          l += p4[j];
        }
        pk[i][kb][0] = bf16_pair_rne(p4[0], p4[1]);
        pk[i][kb][1] = bf16_pair_rne(p4[2], p4[3]);
      }
      lrun[i] = l;
      mrun[i] = mx;
      // scaling by exactly 1 changes nothing: skip it while no lane's max moved
      rescale[i] = __builtin_amdgcn_ballot_w64(alpha[i] != 1.0f) != 0;
    }
    // O^T += V^T P^T: a V^T fragment is read once for all RB blocks
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) {
      f32x4_t acc[RB];
#pragma unroll
      for (int i = 0; i < RB; ++i) acc[i] = rescale[i] ? oacc[i][ob] * alpha[i] : oacc[i][ob];
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2) {
        // A (V^T): dim ob*16 + lq, keys {4 lg .. +3} of block 2 ks2, then of
        // block 2 ks2 + 1; B (P^T): the same keys
        const int vr = ob * 16 + lq;
        const uint16_t *vrow = Vt + vr * VTS;
        const u32x2_t a0 = *reinterpret_cast<const u32x2_t *>(vrow + vt_col(vr, ks2 * 32 + lg * 4));
        const u32x2_t a1 = *reinterpret_cast<const u32x2_t *>(vrow + vt_col(vr, ks2 * 32 + lg * 4 + 16));
        const u32x4_t a = {a0[0], a0[1], a1[0], a1[1]};
#pragma unroll
        for (int i = 0; i < RB; ++i) {
          const u32x4_t b = {pk[i][2 * ks2][0], pk[i][2 * ks2][1], pk[i][2 * ks2 + 1][0], pk[i][2 * ks2 + 1][1]};
          acc[i] = mfma16x16x32(a, b, acc[i]);
        }
      }
#pragma unroll
      for (int i = 0; i < RB; ++i) oacc[i][ob] = acc[i];
    }
    __syncthreads();
  }
  // normalise and store: lane holds dims ob*16 + 4 lg + j of query lq
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    float l = lrun[i];
    l += shfl_xor_f32(l, 16);
    l += shfl_xor_f32(l, 32);
    if (qok[i]) {
      const int h = hrow[i];
      const float inv = F8 ? kv.vs / l : 1.0f / l;
      uint16_t *dst = out + (size_t)(row0 + qrel[i]) * nq * HD + (kh * G + h) * HD + lg * 4;
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        u32x2_t w = {pack_bf16x2(oacc[i][ob][0] * inv, oacc[i][ob][1] * inv),
                     pack_bf16x2(oacc[i][ob][2] * inv, oacc[i][ob][3] * inv)};
        *reinterpret_cast<u32x2_t *>(dst + ob * 16) = w;
      }
    }
  }
}

constexpr float kPrefillSlack = 8.0f;  // log2 units
// V^T swizzle of the 32x32 item: 4-key group g of row r is stored at group
// g ^ s(r), s(r) = bit 4 of r in bit 0 and bits 5-6 of r in bits 2-3.  Rows
// of one 8-row store group share s; with rows of 68 elements the P.V reads
// (row 32 ob + lq, keys 16 k' + 8 h + 4 lh) meet no bank twice, the stores
// two-way at most, and each lane's two key halves h stay in address order,
// so every pair of reads merges into one.
__device__ __forceinline__ int vt32_col(int r, int key) {
  return 4 * ((key >> 2) ^ (((r >> 4) & 1) | (((r >> 5) & 3) << 2))) + (key & 3);
}


// Prefill item on 32x32x16 products: 128 query rows per item (G heads x
// 128 / G positions) over 4 wavefronts, 32 rows (one 32-column block of the
// products) per wave.  Against 16-row blocks every K and V^T fragment read
// from LDS serves twice the rows, so a tile costs half the LDS reads per
// FLOP.  Per 64-key tile a wave forms S^T = K Q^T as two 32-key blocks
// (eight k-steps of 16 dims each), keeps its query's 32 scores in the lane
// pair (l, l + 32), and feeds P^T straight from the score registers into
// O^T += V^T P^T: k-step j of the P.V product takes score values 8 j' ..
// 8 j' + 7 of key block j / 2 (j' = j % 2), i.e. keys 16 j' + {0..3, 8..11}
// + 4 (l / 32) of the block, and the V^T operand reads the same keys.
template <int HD, int G, int NW, bool F8>
__device__ __forceinline__ void prefill_item32(const uint16_t *__restrict__ qkv, int nq, int nkv, const KV kv,
                                               const DevMeta md, int tile, int kh, uint16_t *__restrict__ out,
                                               uint16_t *Ks, uint16_t *Vt) {
  constexpr int BQ = NW * 32 / G;          // query positions per item
  static_assert(NW * 32 == G * BQ, "rows per item");
  constexpr int KT = 64;                   // keys per tile
  constexpr int KSS = HD + 8, VTS = KT + 4;
  constexpr int KCH = KT * (HD / 8), VCH = (KT / 2) * (HD / 8);
  constexpr int NT = NW * 64;
  constexpr int KPT = (KCH + NT - 1) / NT, VPT = (VCH + NT - 1) / NT;
  constexpr int NKS = HD / 16;  // k-steps of the QK^T product
  constexpr int NOB = HD / 32;  // 32-dim output blocks
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cols = (nq + 2 * nkv) * HD;
  // the item's metadata is uniform: held in scalar registers, so that the
  // page arithmetic derived from it stays scalar too
  const int seq = __builtin_amdgcn_readfirstlane(md.tile_seq[tile]);
  const int qb = __builtin_amdgcn_readfirstlane(md.tile_qb[tile]);
  const int c = __builtin_amdgcn_readfirstlane(md.seq_ctx[seq]);
  const int n = __builtin_amdgcn_readfirstlane(md.seq_len[seq]);
  const int row0 = __builtin_amdgcn_readfirstlane(md.seq_row[seq]);
  const int q_lo = qb * BQ;
  const int q_hi = min(n, q_lo + BQ);
  const int kend = c + q_hi;
  const int klen = c + n;
  const int32_t *bt = kv.bt + (size_t)seq * kv.max_pages;
  const int npages = (klen + kPageSize - 1) / kPageSize;
  const float qscale = F8 ? kLog2e / sqrtf((float)HD) * kv.ks : kLog2e / sqrtf((float)HD);
  const int lq = lane & 31;  // query column of this lane
  const int lh = lane >> 5;  // k half

  // the wave's 32 rows: HPB heads x RPH positions
  constexpr int RPH = BQ < 32 ? BQ : 32, HPB = 32 / RPH, HG = G / HPB;
  static_assert(HPB * RPH == 32 && HG * HPB == G, "row block shape");
  const int hb = wave % HG, sub = wave / HG;
  const int hrow = hb * HPB + lq / RPH;
  const int qrel = q_lo + sub * RPH + lq % RPH;
  const bool qok = qrel < q_hi;
  u32x4_t qreg[NKS];
  {
    const uint16_t *src = qkv + (size_t)(row0 + qrel) * cols + (kh * G + hrow) * HD + lh * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qreg[ks] = qok ? ld_u32x4(src + ks * 16) : u32x4_t{0, 0, 0, 0};
  }
  f32x16_t oacc[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[ob][i] = 0.f;
  float mrun = kNegInf, lrun = 0.f;

  typedef int i32x4_t __attribute__((ext_vector_type(4)));
  constexpr int PPT = KT / kPageSize;
  static_assert(PPT == 4, "tile = 4 pages");
  typedef const __attribute__((address_space(4))) int32_t *bt_ptr_t;
  const bt_ptr_t btc = (bt_ptr_t)bt;
  // page ids of tile t; pages past the sequence repeat its last id (their
  // ranges below are empty), so the loads need no branch and no select
  auto bt_tile = [&](int t) -> i32x4_t {
    const int p0 = t * PPT;
    i32x4_t r;
#pragma unroll
    for (int j = 0; j < PPT; ++j) r[j] = btc[min(p0 + j, npages - 1)];
    return r;
  };
  static_assert(HD == 64 || HD == 128, "keys of one load within one page");
  typedef typename std::conditional<F8, const uint8_t, const uint16_t>::type elem_t;
  constexpr int ES = F8 ? 1 : 2;  // bytes per cache element
  // Page j of tile t as a buffer range over its keys below klen (empty for an
  // id outside the pool): loads past it return zeros without memory traffic,
  // so keys past the sequence and bad ids stage as zeros with no selects.
  constexpr uint32_t kPageHeadBytes = kPageSize * HD * ES;
  const uint32_t page_bytes = (uint32_t)nkv * kPageHeadBytes;  // one page of all kv heads
  auto page_rsrc = [&](const uint8_t *base, const i32x4_t &btv, int j, int first_key) -> buf_rsrc_t {
    const int phys = j == 0 ? btv[0] : j == 1 ? btv[1] : j == 2 ? btv[2] : btv[3];
    const int rem = klen - first_key;  // keys of the sequence from the page's first on
    const bool live = (unsigned)phys < (unsigned)kv.num_pages && rem > 0;
    // (uniform; said so, or the compiler forms the range in vector registers
    // and wraps every load in a loop over distinct descriptors)
    const int range = __builtin_amdgcn_readfirstlane(live ? min(rem, kPageSize) * (HD * ES) : 0);
    return make_rsrc(base + (uint64_t)(uint32_t)(live ? phys : 0) * page_bytes, range);
  };
  auto ld8 = [&](buf_rsrc_t r, int off) -> RawT<F8> {
    if constexpr (F8)
      return buf_ld_u32x2<0>(r, off);
    else
      return buf_ld_u32x4<0>(r, off);
  };
  const uint8_t *const kbase = reinterpret_cast<const uint8_t *>(kv.k) + (size_t)kh * kPageHeadBytes;
  const uint8_t *const vbase = reinterpret_cast<const uint8_t *>(kv.v) + (size_t)kh * kPageHeadBytes;
  RawT<F8> kreg[KPT], vreg[VPT][2];
  static_assert(KCH % NT == 0 && VCH % NT == 0, "whole load rounds");
  // round i of the K loads covers keys i * NT / (HD / 8) .. (page fixed per
  // wave); round i of the V loads covers key pairs likewise
  constexpr int KPR = NT / (HD / 8), WPK = kPageSize * (HD / 8) / 64;  // keys per round, waves per page
  static_assert(KPR % kPageSize == 0, "pages per round");
  // the page of K load i: i KPR / 16 + wave / WPK (the second term is 0 when
  // one round covers whole pages per wave group of NW)
  const int kpw = NW <= WPK ? 0 : wave / WPK;
  auto fetch = [&](int t, const i32x4_t &btv) {
    const int k0 = t * KT;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int u = tid + i * NT;
      const int key = u / (HD / 8), dc = u % (HD / 8);
      const int j = i * (KPR / kPageSize) + kpw;
      kreg[i] = ld8(page_rsrc(kbase, btv, j, k0 + j * kPageSize), ((key % kPageSize) * HD + dc * 8) * ES);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      const int kpair = u / (HD / 8), dc = u % (HD / 8);
      const int j = i * (KPR / 8) + wave / (HD / 64);  // page of keys 2 kpair, 2 kpair + 1
      const buf_rsrc_t r = page_rsrc(vbase, btv, j, k0 + j * kPageSize);
#pragma unroll
      for (int e = 0; e < 2; ++e) vreg[i][e] = ld8(r, (((2 * kpair + e) % kPageSize) * HD + dc * 8) * ES);
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int u = tid + i * NT;
      st_u32x4(Ks + (u / (HD / 8)) * KSS + (u % (HD / 8)) * 8, raw_bf16<F8>(kreg[i]));
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const int u = tid + i * NT;
      const int kpair = u / (HD / 8), dc = u % (HD / 8);
      const int col = vt32_col(dc * 8, 2 * kpair);
      const u32x4_t v0 = raw_bf16<F8>(vreg[i][0]), v1 = raw_bf16<F8>(vreg[i][1]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {  // dims 2 j, 2 j + 1 of keys 2 kpair, 2 kpair + 1
        *reinterpret_cast<uint32_t *>(Vt + (dc * 8 + 2 * j) * VTS + col) = __builtin_amdgcn_perm(v1[j], v0[j], 0x05040100u);
        *reinterpret_cast<uint32_t *>(Vt + (dc * 8 + 2 * j + 1) * VTS + col) = __builtin_amdgcn_perm(v1[j], v0[j], 0x07060302u);
      }
    }
  };

  const int min_qpos = c + q_lo;
  const int qpos = c + qrel;
  const int ntiles = (kend + KT - 1) / KT;
  // V^T operand of the P.V product: row ob 32 + lq, keys kb 32 + 16 jj + 8 h
  // + 4 lh .. + 3 at vt32_col(row, key), which splits into a lane part and a
  // constant (the swizzle's lane bit lq / 16 meets only lh, its ob bits only
  // kb and jj), so every read is one base register plus an immediate offset
  static_assert(NOB <= 4, "ob bits of the swizzle");
  const uint16_t *const vlane = Vt + lq * VTS + 4 * (lh ^ (lq >> 4));
  auto vt_at = [&](int ob, int kb, int jj, int h) -> const uint16_t * {
    return vlane + ob * 32 * VTS + 8 * h + 16 * ((2 * kb + jj) ^ ob);
  };
  i32x4_t bt_next = bt_tile(1);
  fetch(0, bt_tile(0));
  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * KT;
    stage();
    __syncthreads();
    // S^T: two 32-key blocks, lane value i at key 32 kb + 8 (i / 4) + 4 lh + i % 4
    f32x16_t sc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sc[kb][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const u32x4_t a = ld_u32x4(Ks + (kb * 32 + lq) * KSS + ks * 16 + lh * 8);
        sc[kb] = mfma32x32x16(a, qreg[ks], sc[kb]);
      }
    {  // the next tile's loads, issued while the products run and in flight
       // while this tile is consumed (past the last tile: empty ranges, no traffic)
      const i32x4_t bt_cur = bt_next;
      bt_next = bt_tile(t + 2);
      fetch(t + 1, bt_cur);
    }
    // causal mask on the diagonal tiles (rows past the item's end are never
    // stored and do not enter another row's arithmetic)
    if (k0 + KT - 1 > min_qpos) {
      const int d = qpos - k0 - 4 * lh;  // value i of block kb is visible iff its key offset is <= d
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[kb][i] = kb * 32 + 8 * (i >> 2) + (i & 3) > d ? kNegInf : sc[kb][i];
    }
    float mraw = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mraw = fmaxf(mraw, sc[kb][i]);
    {  // with the other half of the wave (lane l ^ 32 holds the same query)
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mraw), __float_as_uint(mraw), false, false);
      mraw = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    // The running max (log2 units) moves only when the tile's max exceeds it
    // by more than kPrefillSlack; in between, probabilities stay below
    // 2^kPrefillSlack, exact in fp32 and bf16 alike, and most tiles skip the
    // rescaling of the accumulators.  The normaliser sums the bf16 values
    // that enter the P.V product.
    const float ms = mraw * qscale;
    const bool bump = ms > mrun + kPrefillSlack;
    const float mx = bump ? ms : mrun;
    const float alpha = bump ? fast_exp2(mrun - mx) : 1.0f;  // 0 on the first tile
    const float neg = mx != kNegInf ? -mx : 0.f;
    float l = lrun * alpha;
    uint32_t pk[2][8];  // [key block][pair]: bf16 pairs of values 2 p, 2 p + 1
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int pr = 0; pr < 8; ++pr) {
        const float p0 = fast_exp2(fmaf(sc[kb][2 * pr], qscale, neg));
        const float p1 = fast_exp2(fmaf(sc[kb][2 * pr + 1], qscale, neg));
        pk[kb][pr] = bf16_pair_rne(p0, p1);
        l = dot2_bf16(pk[kb][pr], 0x3F803F80u, l);  // + both values, (1, 1) in bf16
      }
    // (a row whose max was still -inf has nothing accumulated to rescale)
    const bool rescale = __builtin_amdgcn_ballot_w64(bump && mrun != kNegInf) != 0;
    lrun = l;
    mrun = mx;
    if (__builtin_expect(rescale, 0)) {
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) oacc[ob] = oacc[ob] * alpha;
    }
    // O^T += V^T P^T: k-step j takes keys 16 (j % 2) + {0..3, 8..11} + 4 lh of key block j / 2
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) {
      f32x16_t acc = oacc[ob];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kb = j >> 1, jj = j & 1;
        const u32x2_t a0 = *reinterpret_cast<const u32x2_t *>(vt_at(ob, kb, jj, 0));
        const u32x2_t a1 = *reinterpret_cast<const u32x2_t *>(vt_at(ob, kb, jj, 1));
        const u32x4_t a = {a0[0], a0[1], a1[0], a1[1]};
        const u32x4_t b = {pk[kb][4 * jj], pk[kb][4 * jj + 1], pk[kb][4 * jj + 2], pk[kb][4 * jj + 3]};
        acc = mfma32x32x16(a, b, acc);
      }
      oacc[ob] = acc;
    }
    __syncthreads();
  }
  // normalise and store: lane holds dims ob 32 + 8 g + 4 lh + e (e < 4) of its query
  float l = lrun;
  l += shfl_xor_f32(l, 32);
  if (qok) {
    const float inv = F8 ? kv.vs / l : 1.0f / l;
    uint16_t *dst = out + (size_t)(row0 + qrel) * nq * HD + (kh * G + hrow) * HD + 4 * lh;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2_t w = {pack_bf16x2(oacc[ob][4 * g] * inv, oacc[ob][4 * g + 1] * inv),
                           pack_bf16x2(oacc[ob][4 * g + 2] * inv, oacc[ob][4 * g + 3] * inv)};
        *reinterpret_cast<u32x2_t *>(dst + ob * 32 + 8 * g) = w;
      }
  }
}

// One 16-byte-per-lane load from a buffer range straight into LDS: lane l
// fills bytes 16 l .. 16 l + 15 from dst (wave-uniform) with the bytes at its
// offset (zeros past the range).
__device__ __forceinline__ void lds_dma16(buf_rsrc_t r, uint8_t *dst, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t *)dst, 16, off, 0, 0, 0);
}

// The 32x32 prefill item for bf16 caches with its tiles loaded straight
// into LDS: two buffers of a K tile and a V tile (64 keys x HD, row-major,
// 16-byte chunks swizzled), the next tile's loads issued at the top of a
// tile and landed by the barrier that ends it, so there is no register
// staging and one barrier per tile.  The scores read K chunks as in
// prefill_item32; the P.V product reads its V^T operand with the transposing
// LDS read (ds_read_b64_tr_b16: within 16 lanes, lane i receives element
// i % 4 of the 8-byte pieces that lanes 4 e + i / 4 point at, e = 0..3), so
// each lane gets one dim of four keys and V needs no transpose on its way in.
// Chunk swizzles: K chunk c of key t sits at position c ^ (t & 7), so the 8
// rows of one pass of a 16-byte read start in 8 bank groups; V chunk c of
// key t at c ^ 2 (t & 3), so the 4 keys x 2 chunks of a transposed read's 16
// lanes fall in 8 bank groups.
template <int HD, int G, int NW>
__device__ __forceinline__ void prefill_item32_dma(const uint16_t *__restrict__ qkv, int nq, int nkv, const KV kv,
                                                   const DevMeta md, int tile, int kh, uint16_t *__restrict__ out,
                                                   uint8_t *buf0, uint8_t *buf1) {
  constexpr int BQ = NW * 32 / G;  // query positions per item
  static_assert(NW * 32 == G * BQ, "rows per item");
  constexpr int KT = 64;                 // keys per tile
  constexpr int ROW = HD * 2;            // bytes per key row
  constexpr int CPR = ROW / 16;          // 16-byte chunks per row
  constexpr int TILE = KT * ROW;         // bytes of the K (and of the V) tile
  constexpr int KPI = 1024 / ROW;        // keys per 1 KiB load instruction
  constexpr int NI = KT / (KPI * NW);    // load instructions per wave per tile, each of K and V
  static_assert(NI * KPI * NW == KT && KPI <= kPageSize, "whole load rounds within pages");
  constexpr int NKS = HD / 16;  // k-steps of the QK^T product
  constexpr int NOB = HD / 32;  // 32-dim output blocks
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int cols = (nq + 2 * nkv) * HD;
  const int seq = __builtin_amdgcn_readfirstlane(md.tile_seq[tile]);
  const int qb = __builtin_amdgcn_readfirstlane(md.tile_qb[tile]);
  const int c = __builtin_amdgcn_readfirstlane(md.seq_ctx[seq]);
  const int n = __builtin_amdgcn_readfirstlane(md.seq_len[seq]);
  const int row0 = __builtin_amdgcn_readfirstlane(md.seq_row[seq]);
  const int q_lo = qb * BQ;
  const int q_hi = min(n, q_lo + BQ);
  const int kend = c + q_hi;
  const int klen = c + n;
  const int32_t *bt = kv.bt + (size_t)seq * kv.max_pages;
  const int npages = (klen + kPageSize - 1) / kPageSize;
  const float qscale = kLog2e / sqrtf((float)HD);
  const int lq = lane & 31;  // query column of this lane
  const int lh = lane >> 5;  // k half

  // the wave's 32 rows: HPB heads x RPH positions
  constexpr int RPH = BQ < 32 ? BQ : 32, HPB = 32 / RPH, HG = G / HPB;
  static_assert(HPB * RPH == 32 && HG * HPB == G, "row block shape");
  const int hb = wave % HG, sub = wave / HG;
  const int hrow = hb * HPB + lq / RPH;
  const int qrel = q_lo + sub * RPH + lq % RPH;
  const bool qok = qrel < q_hi;
  u32x4_t qreg[NKS];
  {
    const uint16_t *src = qkv + (size_t)(row0 + qrel) * cols + (kh * G + hrow) * HD + lh * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qreg[ks] = qok ? ld_u32x4(src + ks * 16) : u32x4_t{0, 0, 0, 0};
  }
  f32x16_t oacc[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[ob][i] = 0.f;
  float mrun = kNegInf, lrun = 0.f;

  typedef int i32x4_t __attribute__((ext_vector_type(4)));
  constexpr int PPT = KT / kPageSize;
  static_assert(PPT == 4, "tile = 4 pages");
  typedef const __attribute__((address_space(4))) int32_t *bt_ptr_t;
  const bt_ptr_t btc = (bt_ptr_t)bt;
  auto bt_tile = [&](int t) -> i32x4_t {  // pages past the sequence repeat its last id (empty ranges below)
    const int p0 = t * PPT;
    i32x4_t r;
#pragma unroll
    for (int j = 0; j < PPT; ++j) r[j] = btc[min(p0 + j, npages - 1)];
    return r;
  };
  constexpr uint32_t kPageHeadBytes = kPageSize * ROW;
  const uint32_t page_bytes = (uint32_t)nkv * kPageHeadBytes;
  const uint8_t *const kbase = reinterpret_cast<const uint8_t *>(kv.k) + (size_t)kh * kPageHeadBytes;
  const uint8_t *const vbase = reinterpret_cast<const uint8_t *>(kv.v) + (size_t)kh * kPageHeadBytes;
  // page j of a tile as a buffer range over its keys below klen (empty for
  // an id outside the pool): loads past it land as zeros, without traffic
  auto page_rsrc = [&](const uint8_t *base, const i32x4_t &btv, int j, int first_key) -> buf_rsrc_t {
    const int phys = j == 0 ? btv[0] : j == 1 ? btv[1] : j == 2 ? btv[2] : btv[3];
    const int rem = klen - first_key;
    const bool live = (unsigned)phys < (unsigned)kv.num_pages && rem > 0;
    const int range = __builtin_amdgcn_readfirstlane(live ? min(rem, kPageSize) * ROW : 0);
    return make_rsrc(base + (uint64_t)(uint32_t)(live ? phys : 0) * page_bytes, range);
  };
  // load instruction i of wave w fills keys KPI (i NW + w) .. + KPI - 1 of a
  // tile; lane l writes chunk position l % CPR of key KPI (i NW + w) + l / CPR
  uint32_t koff[NI], voff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int key = KPI * (i * NW + wave) + lane / CPR;  // within the tile
    const int pos = lane % CPR;
    koff[i] = (uint32_t)((key % kPageSize) * ROW + 16 * (pos ^ (key & 7)));
    voff[i] = (uint32_t)((key % kPageSize) * ROW + 16 * (pos ^ (2 * (key & 3))));
  }
  // the K (or V) tile of tile t into dst
  auto dma = [&](int t, const i32x4_t &btv, uint8_t *dst, bool is_v) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int key0 = KPI * (i * NW + wave);
      const int j = key0 / kPageSize;  // wave-uniform
      const int first = t * KT + j * kPageSize;
      lds_dma16(page_rsrc(is_v ? vbase : kbase, btv, j, first), dst + key0 * ROW, is_v ? voff[i] : koff[i]);
    }
  };

  // K operand of the scores: key kb 32 + lq, chunk 2 ks + lh at position
  // (2 ks + lh) ^ (lq & 7) (bit 3 of the chunk, ks >> 2, is untouched)
  int kaddr[4];
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) kaddr[k4] = lq * ROW + 16 * ((2 * k4 + lh) ^ (lq & 7));
  // V^T operand, the transposed read: lane 16 g + 4 e + q points at key
  // kb 32 + 16 jj + 8 h + 4 (g / 2) + e, dims ob 32 + 16 (g & 1) + 4 q .. + 3,
  // i.e. chunk 4 ob + 2 (g & 1) + q / 2 (half q & 1) at position
  // chunk ^ 2 e; the lane part depends on ob & 1 only
  const int tg = lane >> 4, te = (lane >> 2) & 3, tq = lane & 3;
  int vaddr[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
    vaddr[b] = (4 * (tg >> 1) + te) * ROW + 16 * ((4 * b + 2 * (tg & 1) + (tq >> 1)) ^ (2 * te)) + 8 * (tq & 1);
  typedef short v4s_t __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;
  auto vt_read = [&](const uint8_t *vt, int ob, int kb, int jj, int h) -> u32x2_t {
    const uint8_t *p = vt + vaddr[ob & 1] + (kb * 32 + 16 * jj + 8 * h) * ROW + 128 * (ob >> 1);
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t *)p));
  };

  const int min_qpos = c + q_lo;
  const int qpos = c + qrel;
  const int ntiles = (kend + KT - 1) / KT;
  // S^T of the K tile at kt: two 32-key blocks, lane value i at key
  // 32 kb + 8 (i / 4) + 4 lh + i % 4
  auto scores = [&](const uint8_t *kt, f32x16_t (&s)[2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const u32x4_t a = *reinterpret_cast<const u32x4_t *>(kt + kaddr[ks & 3] + 128 * (ks >> 2) + kb * 32 * ROW);
        s[kb] = mfma32x32x16(a, qreg[ks], s[kb]);
      }
  };
  // Buffer b holds K tile and V tile of tiles b, b + 2, ...  K goes two tiles
  // ahead and V one, so during tile t the scores of tile t + 1 (K landed by
  // the barrier that ended tile t - 1) are formed while tile t's softmax
  // runs: the two are independent and the matrix products overlap the
  // exponentials.  One barrier per tile lands the loads issued at its top
  // (K of t + 2, V of t + 1) and retires every read of the buffers they
  // refill.
  f32x16_t sc[2];
  i32x4_t bt1 = bt_tile(1), bt2 = bt_tile(2);
  dma(0, bt_tile(0), buf0, false);
  dma(0, bt_tile(0), buf0 + TILE, true);
  if (ntiles > 1) dma(1, bt1, buf1, false);
  __syncthreads();
  scores(buf0, sc);
  __syncthreads();  // every wave past the scores of tile 0 before K of tile 2 refills buffer 0
  auto step = [&](int t, auto lastconst) {
    constexpr bool LAST = decltype(lastconst)::value;
    uint8_t *const cur = (t & 1) ? buf1 : buf0, *const nxt = (t & 1) ? buf0 : buf1;
    const int k0 = t * KT;
    f32x16_t scn[2];
    if constexpr (!LAST) {
      if (t + 2 < ntiles) dma(t + 2, bt2, cur, false);  // K of tile t was read by its scores before the last barrier
      dma(t + 1, bt1, nxt + TILE, true);                // V of tile t - 1 was read before the last barrier
      bt1 = bt2;
      bt2 = bt_tile(t + 3);
    }
    if (k0 + KT - 1 > min_qpos) {  // causal mask on the diagonal tiles
      const int d = qpos - k0 - 4 * lh;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) sc[kb][i] = kb * 32 + 8 * (i >> 2) + (i & 3) > d ? kNegInf : sc[kb][i];
    }
    if constexpr (!LAST) scores(nxt, scn);
    float mraw = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mraw = fmaxf(mraw, sc[kb][i]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mraw), __float_as_uint(mraw), false, false);
      mraw = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    }
    // lazy running max and bf16 normaliser, as in prefill_item32
    const float ms = mraw * qscale;
    const bool bump = ms > mrun + kPrefillSlack;
    const float mx = bump ? ms : mrun;
    const float alpha = bump ? fast_exp2(mrun - mx) : 1.0f;
    const float neg = mx != kNegInf ? -mx : 0.f;
    float l = lrun * alpha;
    uint32_t pk[2][8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int pr = 0; pr < 8; ++pr) {
        const float p0 = fast_exp2(fmaf(sc[kb][2 * pr], qscale, neg));
        const float p1 = fast_exp2(fmaf(sc[kb][2 * pr + 1], qscale, neg));
        pk[kb][pr] = bf16_pair_rne(p0, p1);
        l = dot2_bf16(pk[kb][pr], 0x3F803F80u, l);
      }
    // (the test on l, true for every finite sum, ties the branch below to
    // the block above: decided earlier, it would split that block and keep
    // the score products from running under the exponentials)
    const bool rescale = __builtin_amdgcn_ballot_w64(bump && mrun != kNegInf && l >= 0.f) != 0;
    lrun = l;
    mrun = mx;
    if (__builtin_expect(rescale, 0)) {
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) oacc[ob] = oacc[ob] * alpha;
    }
    // O^T += V^T P^T: k-step j takes keys 16 (j % 2) + {0..3, 8..11} + 4 lh of key block j / 2
    const uint8_t *const vt = cur + TILE;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) {
      f32x16_t acc = oacc[ob];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kb = j >> 1, jj = j & 1;
        const u32x2_t a0 = vt_read(vt, ob, kb, jj, 0), a1 = vt_read(vt, ob, kb, jj, 1);
        const u32x4_t a = {a0[0], a0[1], a1[0], a1[1]};
        const u32x4_t b = {pk[kb][4 * jj], pk[kb][4 * jj + 1], pk[kb][4 * jj + 2], pk[kb][4 * jj + 3]};
        acc = mfma32x32x16(a, b, acc);
      }
      oacc[ob] = acc;
    }
    if constexpr (!LAST) {
      sc[0] = scn[0];
      sc[1] = scn[1];
      __syncthreads();
    }
  };
  for (int t = 0; t + 1 < ntiles; ++t) step(t, std::false_type{});
  step(ntiles - 1, std::true_type{});
  float l = lrun;
  l += shfl_xor_f32(l, 32);
  if (qok) {
    const float inv = 1.0f / l;
    uint16_t *dst = out + (size_t)(row0 + qrel) * nq * HD + (kh * G + hrow) * HD + 4 * lh;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2_t w = {pack_bf16x2(oacc[ob][4 * g] * inv, oacc[ob][4 * g + 1] * inv),
                           pack_bf16x2(oacc[ob][4 * g + 2] * inv, oacc[ob][4 * g + 3] * inv)};
        *reinterpret_cast<u32x2_t *>(dst + ob * 32 + 8 * g) = w;
      }
  }
}

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------
// Work item of block b in a launch of n blocks (decode units, or the mixed
// launch's interleaved items).  Consecutive decode units are the kv heads of
// one split, which read the same pages (each page holds every
// head's keys of its 16 positions), and blocks are dealt round-robin to the
// 8 XCDs; so within each run of 64 blocks, block b takes item
// 8 (b % 8) + (b % 64) / 8 of the run, which puts each 8 consecutive items
// on one XCD, whose L2 and address translation then serve a page for all
// its heads.  The order of the runs is kept; a last run shorter than 64
// keeps the identity.
__device__ __forceinline__ int xcd_grouped_unit(int b, int n) {
  if (b >= (n & ~63)) return b;
  return (b & ~63) + ((b & 7) << 3) + ((b & 63) >> 3);
}

template <int HD, int G, bool F8>
__global__ __launch_bounds__(256, 2) void k_decode(const uint16_t *qkv, int nq, int nkv, KV kv, DevMeta md,
                                                   uint16_t *out, float *part_o, float *part_ml) {
  __shared__ float lds[DecodeTraits<HD, G, 4>::LDS_BYTES / 4];
  decode_item<HD, G, 4, F8>(qkv, nq, nkv, kv, md, xcd_grouped_unit(blockIdx.x, gridDim.x), out, part_o, part_ml, lds);
}

// The matrix-core decode keeps its page slots in separate LDS arrays, so the
// compiler's wait before reading one slot covers only that slot's loads.
// Decode-only launch: kDecWaves wavefronts per block, rings kDecSlots deep
// for bf16 pages and kDecSlotsF8 deep for 8-bit ones (a slot sized to the
// page, half the bf16 one).
constexpr int kDecWaves = 4, kDecSlots = 2, kDecSlotsF8 = 2;
#define EB_MDEC_LDS(ARRAY_, NSLOT_)                                                  \
  __shared__ __attribute__((aligned(16))) uint8_t l0[ARRAY_];                        \
  __shared__ __attribute__((aligned(16))) uint8_t l1[ARRAY_];                        \
  __shared__ __attribute__((aligned(16))) uint8_t l2[NSLOT_ > 2 ? (ARRAY_) : 16];    \
  __shared__ __attribute__((aligned(16))) uint8_t l3[NSLOT_ > 3 ? (ARRAY_) : 16];

// 8-bit pages: four blocks per CU (LDS 4 x 32 KiB), so at most 128 registers
template <int HD, int G, bool F8>
__global__ __launch_bounds__(64 * kDecWaves, F8 ? 4 : 1) void k_decode_mfma(const uint16_t *qkv, int nq, int nkv, KV kv,
                                                                DevMeta md, uint16_t *out, float *part_o,
                                                                float *part_ml) {
  constexpr int NS = F8 ? kDecSlotsF8 : kDecSlots;
  constexpr int SLOT = MdecTraits<HD, F8>::SLOT;
  EB_MDEC_LDS(kDecWaves * SLOT, NS)
  decode_item_mfma<HD, G, kDecWaves, NS, F8, SLOT>(qkv, nq, nkv, kv, md, xcd_grouped_unit(blockIdx.x, gridDim.x), out,
                                                   part_o, part_ml, l0, l1, l2, l3);
}

// Prefill-only launch: 4 wavefronts per 128-row item, 32 rows per wave on
// 32x32x16 products.
constexpr int kPrefillWaves = 4;
template <int HD>
struct PrefillLds {
  static constexpr int K_BYTES = 64 * (HD + 8) * 2;  // K tile, row-major
  static constexpr int VT_BYTES = HD * (64 + 4) * 2;  // V^T tile
  static constexpr int DMA_BYTES = 2 * 2 * 64 * HD * 2;  // bf16 caches: two buffers of a K and a V tile
};

template <int HD, int G, bool F8>
__global__ __launch_bounds__(64 * kPrefillWaves, 2) void k_prefill(const uint16_t *qkv, int nq, int nkv, KV kv,
                                                                      DevMeta md, uint16_t *out) {
  constexpr int LB = F8 ? PrefillLds<HD>::K_BYTES + PrefillLds<HD>::VT_BYTES : PrefillLds<HD>::DMA_BYTES;
  __shared__ __attribute__((aligned(16))) uint16_t lds[LB / 2];
  const int item = blockIdx.x / nkv, kh = blockIdx.x % nkv;
  if constexpr (F8) {
    prefill_item32<HD, G, kPrefillWaves, F8>(qkv, nq, nkv, kv, md, item, kh, out, lds, lds + PrefillLds<HD>::K_BYTES / 2);
  } else {
    uint8_t *const b0 = reinterpret_cast<uint8_t *>(lds);
    prefill_item32_dma<HD, G, kPrefillWaves>(qkv, nq, nkv, kv, md, item, kh, out, b0,
                                             b0 + PrefillLds<HD>::DMA_BYTES / 2);
  }
}

// One grid for a mixed step: items [0, n_tiles) are prefill tiles (longest
// first), the rest decode splits; every block (4 wavefronts) branches
// uniformly on its kind.  Decode items run exactly the decode-only code.
// Block b of a mixed launch: prefill item (>= 0) or decode unit (the
// complement), from the interleaving stride s (see mixed_prefill_stride).
__device__ __forceinline__ void mixed_slot(int b, int n_prefill, int s, int &pf, int &du) {
  const int q = b / s;
  if (b - q * s == 0 && q < n_prefill) {
    pf = q;
    du = -1;
  } else {
    pf = -1;
    du = b - min(n_prefill, q + 1);
  }
}

template <int HD, int G, bool F8>
__global__ __launch_bounds__(256, 2) void k_mixed(const uint16_t *qkv, int nq, int nkv, KV kv, DevMeta md, uint16_t *out,
                                               float *part_o, float *part_ml, int stride) {
  constexpr int PB = F8 ? PrefillLds<HD>::K_BYTES + PrefillLds<HD>::VT_BYTES : PrefillLds<HD>::DMA_BYTES;
  constexpr int DB = DecodeTraits<HD, G, 4>::LDS_BYTES;
  __shared__ __attribute__((aligned(16))) uint16_t lds[(PB > DB ? PB : DB) / 2];
  int pf, du;
  mixed_slot(xcd_grouped_unit(blockIdx.x, gridDim.x), md.n_tiles * nkv, stride, pf, du);
  if (pf >= 0) {
    if constexpr (F8)
      prefill_item32<HD, G, 4, F8>(qkv, nq, nkv, kv, md, pf / nkv, pf % nkv, out, lds,
                                   lds + PrefillLds<HD>::K_BYTES / 2);
    else
      prefill_item32_dma<HD, G, 4>(qkv, nq, nkv, kv, md, pf / nkv, pf % nkv, out, reinterpret_cast<uint8_t *>(lds),
                                   reinterpret_cast<uint8_t *>(lds) + PrefillLds<HD>::DMA_BYTES / 2);
  } else
    decode_item<HD, G, 4, F8>(qkv, nq, nkv, kv, md, du, out, part_o, part_ml, reinterpret_cast<float *>(lds));
}

// The same with matrix-core decode items; prefill tiles borrow two of the
// page-slot arrays.
template <int HD, int G, bool F8>
__global__ __launch_bounds__(256, 2) void k_mixed_mfma(const uint16_t *qkv, int nq, int nkv, KV kv, DevMeta md,
                                                    uint16_t *out, float *part_o, float *part_ml, int stride) {
  constexpr int MS = 2;                           // ring depth of decode items in the mixed launch
  constexpr int SLOT = MdecTraits<HD>::SLOT;      // bf16-sized slots: prefill tiles stage bf16
  static_assert(PrefillLds<HD>::K_BYTES <= 4 * SLOT && PrefillLds<HD>::VT_BYTES <= 4 * SLOT &&
                    PrefillLds<HD>::DMA_BYTES / 2 <= 4 * SLOT, "LDS");
  EB_MDEC_LDS(4 * SLOT, MS)
  int pf, du;
  mixed_slot(xcd_grouped_unit(blockIdx.x, gridDim.x), md.n_tiles * nkv, stride, pf, du);
  if (pf >= 0) {
    if constexpr (F8)
      prefill_item32<HD, G, 4, F8>(qkv, nq, nkv, kv, md, pf / nkv, pf % nkv, out, reinterpret_cast<uint16_t *>(l0),
                                   reinterpret_cast<uint16_t *>(l1));
    else  // one tile buffer in each of the first two page-slot arrays
      prefill_item32_dma<HD, G, 4>(qkv, nq, nkv, kv, md, pf / nkv, pf % nkv, out, l0, l1);
  } else
    decode_item_mfma<HD, G, 4, MS, F8, SLOT>(qkv, nq, nkv, kv, md, du, out, part_o, part_ml, l0, l1, l2, l3);
}
#undef EB_MDEC_LDS

template <int HD, int G, bool F8>
static hipError_t launch_attention_t(const Shape &s, const uint16_t *qkv, const KV &kv, const DevMeta &m,
                                     uint16_t *out, float *part_o, float *part_ml, int kind, int parts,
                                     hipStream_t st) {
  const int nkv = s.nkv, nq = s.nq;
  const bool has_dec = m.n_dec > 0, has_pf = m.n_tiles > 0;
  if (!(parts & 1)) {
    // combine only
  } else if (kind == 2 && has_dec && has_pf) {
    const int stride = mixed_prefill_stride((long)m.n_tiles * nkv, m.total_units);
    if constexpr (kDecodeMfma<G>)
      hipLaunchKernelGGL((k_mixed_mfma<HD, G, F8>), dim3(m.n_tiles * nkv + m.total_units), dim3(256), 0, st, qkv, nq,
                         nkv, kv, m, out, part_o, part_ml, stride);
    else
      hipLaunchKernelGGL((k_mixed<HD, G, F8>), dim3(m.n_tiles * nkv + m.total_units), dim3(256), 0, st, qkv, nq, nkv,
                         kv, m, out, part_o, part_ml, stride);
  } else {
    if (has_pf)
      hipLaunchKernelGGL((k_prefill<HD, G, F8>), dim3(m.n_tiles * nkv), dim3(64 * kPrefillWaves), 0, st, qkv, nq, nkv,
                         kv, m, out);
    if (has_dec) {
      if constexpr (kDecodeMfma<G>)
        hipLaunchKernelGGL((k_decode_mfma<HD, G, F8>), dim3(m.total_units), dim3(64 * kDecWaves), 0, st, qkv, nq, nkv,
                           kv, m, out, part_o, part_ml);
      else
        hipLaunchKernelGGL((k_decode<HD, G, F8>), dim3(m.total_units), dim3(256), 0, st, qkv, nq, nkv, kv, m, out,
                           part_o, part_ml);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((parts & 2) && m.n_comb > 0)
    hipLaunchKernelGGL((k_decode_combine<HD, G>), dim3(m.n_comb, nq), dim3(64), 0, st, m, part_o, part_ml, out, nq, nkv);
  return hipGetLastError();
}

hipError_t launch_attention(const Shape &s, const uint16_t *qkv, const KV &kv, const DevMeta &m, uint16_t *out,
                            float *part_o, float *part_ml, int kind, hipStream_t st, int parts) {
  const int G = s.group();
#define EB_ATT_CASE(HD_, G_)                                                                                 \
  if (s.hd == HD_ && G == G_)                                                                                \
    return kv.f8 ? launch_attention_t<HD_, G_, true>(s, qkv, kv, m, out, part_o, part_ml, kind, parts, st)   \
                 : launch_attention_t<HD_, G_, false>(s, qkv, kv, m, out, part_o, part_ml, kind, parts, st);
  EB_ATT_CASE(128, 1) EB_ATT_CASE(128, 2) EB_ATT_CASE(128, 4) EB_ATT_CASE(128, 8)
  EB_ATT_CASE(64, 1) EB_ATT_CASE(64, 2) EB_ATT_CASE(64, 4) EB_ATT_CASE(64, 8)
#undef EB_ATT_CASE
  return hipErrorInvalidValue;
}

}  // namespace eb
