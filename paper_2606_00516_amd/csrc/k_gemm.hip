// Projection GEMMs of the layer: out = epilogue(A W^T), A [M, K] activations,
// W [N, K] weights, both K-contiguous bf16, fp32 accumulation on the
// 16x16x32 bf16 MFMA.
//
//  * skinny: decode-sized batches (up to 256 rows, 64-row x 128-column
//    tiles, one block per CU).  The product is bound by streaming W from HBM
//    once: tiles stage W and A through LDS in 128-wide K slices read as
//    whole 256-byte rows, the 4 waves of a block own 32 columns each, the
//    row blocks of a column tile run side by side on one XCD so W comes from
//    HBM once, and blocks may further split K, with a small reduction kernel
//    applying the epilogue.
//  * tiled: larger M.  128x128 output tiles, K tiles of 64 double-buffered in
//    LDS, 4 waves each owning a 64x64 sub-tile.
//
// Epilogues: store; + residual; SiLU(gate) * up.  For SiLU the columns are
// processed in groups of 64 = 32 gate rows of W followed by the 32 matching
// up rows (gate rows 0..F-1, up rows F..2F-1 of W), so that every lane holds
// a gate accumulator and its up partner.
#include "device_common.h"
#include "eb_internal.h"

namespace eb {

// W row feeding logical column c of the product (or -1 if none).
__device__ __forceinline__ int w_row_of(int c, int N, int epi) {
  if (epi != EPI_SILU_MUL) return c < N ? c : -1;
  const int F = N >> 1;
  const int g = c >> 6, w = c & 63;
  const int f = g * 32 + (w & 31);
  if (f >= F) return -1;
  return w < 32 ? f : F + f;
}

// Number of logical product columns for an epilogue.
__host__ __device__ static inline int logical_cols(int N, int epi) {
  if (epi != EPI_SILU_MUL) return N;
  const int F = N / 2;
  return ((F + 31) / 32) * 64;
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// 8-bit weights: the fp32 sums of logical columns c .. c + 3 (one W row
// each, consecutive within a column group) times their rows' scales.
__device__ __forceinline__ f32x4_t row_scaled(f32x4_t v, const float *__restrict__ wscale, int c, int N, int epi) {
  const int wr = w_row_of(c, N, epi);
  if (wr < 0) return v;
  const f32x4_t s = *reinterpret_cast<const f32x4_t *>(wscale + wr);
  return v * s;
}

// ===========================================================================
// skinny
// ===========================================================================
constexpr int SK_BN = 64;                // logical columns per block
constexpr int SK_BM = 64;                // rows per block
constexpr int SK_KC = 128;               // K per stage
constexpr int SK_ROWB = SK_KC * 2 + 16;  // LDS bytes per tile row (padded)
constexpr int SK_LDS = 2 * (SK_BN + SK_BM) * SK_ROWB;

// Logical column (0..63 in the block) of row j (0..15) of wave w's slice:
// columns 8w..8w+7 and 32+8w..32+8w+7, so that a SiLU group's gate column
// and its up partner (32 apart) land in the same wave.
__device__ __forceinline__ int sk_col(int w, int j) { return j < 8 ? 8 * w + j : 32 + 8 * w + (j - 8); }

// The weight-streaming kernel's block is 128 logical columns x 64 rows, one
// block per CU.  W and A are staged through LDS in 128-wide K slices (each
// load instruction reads 4 rows x 256 contiguous bytes, so a wave's loads
// touch few pages), and each of the 4 waves owns 32 columns: per K step of
// 32 it reads 2 W and 4 A fragments from LDS for 8 products, so the LDS
// carries 3.5 bytes per weight byte (staging writes included) where a
// 64-column block with 16 columns per wave carried 7.
constexpr int SW_BN = 128;                                 // logical columns per block
constexpr int SW_LDS = 2 * (SW_BN + SK_BM) * SK_ROWB;      // two stages of [128 W rows + 64 A rows]

// Block-local logical column of row lr (0..15) of wave w's column fragment
// f (0, 1): wave w takes half w % 2 of SiLU group w / 2, fragment 0 its 16
// gate columns and fragment 1 their 16 up partners (32 further), so a lane
// holds a gate sum and its partner.
__device__ __forceinline__ int sw_col(int w, int f, int lr) { return (w >> 1) * 64 + f * 32 + (w & 1) * 16 + lr; }

// PRENORM (split-K partials only): A holds the rows x of an RMSNorm that
// precedes the product.  The kernel stages bf16(x * gamma) instead of A and
// the blocks of the first column tile write each row's partial sum of
// squares over their K range to ssq[split][M]; the row scale
// 1 / sqrt(mean(x^2) + eps) is applied to the summed partials by the
// consumer (RMSNorm(x) g W^T = inv * ((x g) W^T)).
template <bool W8, bool PRENORM = false>
__global__ __launch_bounds__(256) void k_gemm_skinny(const uint16_t *__restrict__ A, const void *__restrict__ W,
                                                     const float *__restrict__ wscale, uint16_t *__restrict__ out,
                                                     const uint16_t *__restrict__ res, float *__restrict__ part, int M,
                                                     int N, int K, int epi, int ksteps_per_split, int tiles, int mt,
                                                     int per_xcd, const uint16_t *__restrict__ gamma = nullptr,
                                                     float *__restrict__ ssq = nullptr) {
  extern __shared__ __attribute__((aligned(16))) uint8_t sk_lds[];  // [2][128 W rows + 64 A rows][SK_ROWB]
  // block b takes tile (b % 8) * per_xcd + b / 8, so each XCD walks its own
  // contiguous tile range; the mt row blocks of one column tile are
  // neighbours there and share the W tile through that XCD's L2
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= tiles) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = (t / mt) * SW_BN;
  const int split = blockIdx.y;
  const int m0 = (t % mt) * SK_BM;
  const int kbeg = split * ksteps_per_split * 32;
  const int kend = min(K, kbeg + ksteps_per_split * 32);
  const int nst = kend > kbeg ? (kend - kbeg + SK_KC - 1) / SK_KC : 0;
  constexpr uint32_t WES = W8 ? 1u : 2u;  // bytes per W element
  const buf_rsrc_t ra = make_rsrc(A, (int)min((size_t)M * K * 2, (size_t)0x7FFFFFFF));
  const buf_rsrc_t rw = make_rsrc(W, (int)min((size_t)N * K * WES, (size_t)0x7FFFFFFF));

  // Staging: thread t moves 16-byte chunk t % 16 of W tile rows t / 16 + 16 j
  // (j < 8) and A tile rows t / 16 + 16 j (j < 4); each wave instruction
  // reads 4 rows x 256 contiguous bytes.  Rows outside the operands, k past
  // the block's range: offsets past the descriptor's range, loaded as zero
  // without memory traffic.
  const int ch = tid & 15, r0 = tid >> 4;
  uint32_t woff[8], aoff[4];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int wr = w_row_of(n0 + r0 + 16 * j, N, epi);
    woff[j] = wr >= 0 ? ((uint32_t)wr * (uint32_t)K + (uint32_t)(ch * 8)) * WES : 0x80000000u;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + r0 + 16 * j;
    aoff[j] = m < M ? ((uint32_t)m * (uint32_t)K + (uint32_t)(ch * 8)) * 2u : 0x80000000u;
  }
  u32x4_t wa[8], aa[4], wb[8], ab[4];
  u32x4_t ga = {0u, 0u, 0u, 0u}, gb = {0u, 0u, 0u, 0u};  // PRENORM: gamma chunk of each stage
  float ssacc[4] = {0.f, 0.f, 0.f, 0.f};                 // PRENORM: sum of squares of rows r0 + 16 j
  const buf_rsrc_t rg = make_rsrc(PRENORM ? gamma : A, PRENORM ? K * 2 : 16);
  auto gload = [&](int s, u32x4_t (&wr)[8], u32x4_t (&ar)[4], u32x4_t &gr) {
    const int k = kbeg + s * SK_KC + ch * 8;
    const bool ok = s < nst && k < kend;
    const uint32_t kb = (uint32_t)(kbeg + s * SK_KC) * 2u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if constexpr (W8) {  // 8 codes in the low half; exact bf16 images when staged
        const u32x2_t c = buf_ld_u32x2<kAuxNT>(rw, (int)(ok ? woff[j] + kb / 2u : 0x80000000u));
        wr[j] = u32x4_t{c[0], c[1], 0u, 0u};
      } else {
        wr[j] = buf_ld_u32x4<kAuxNT>(rw, (int)(ok ? woff[j] + kb : 0x80000000u));
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) ar[j] = buf_ld_u32x4<0>(ra, (int)(ok ? aoff[j] + kb : 0x80000000u));
    if constexpr (PRENORM) gr = buf_ld_u32x4<0>(rg, (int)(ok ? (uint32_t)(k * 2) : 0x80000000u));
  };
  const bool first_col_tile = n0 == 0;
  auto swrite = [&](int buf, const u32x4_t (&wr)[8], const u32x4_t (&ar)[4], const u32x4_t &gr) {
    uint8_t *b = sk_lds + buf * (SW_BN + SK_BM) * SK_ROWB;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      u32x4_t wv = wr[j];
      if constexpr (W8) wv = e4m3x8_to_bf16x8(u32x2_t{wr[j][0], wr[j][1]});
      *reinterpret_cast<u32x4_t *>(b + (r0 + 16 * j) * SK_ROWB + ch * 16) = wv;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x4_t av = ar[j];
      if constexpr (PRENORM) {
        if (first_col_tile) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float lo = bf16_lo(ar[j][e]), hi = bf16_hi(ar[j][e]);
            ssacc[j] += lo * lo + hi * hi;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          av[e] = bf16_pair_rne(bf16_lo(ar[j][e]) * bf16_lo(gr[e]), bf16_hi(ar[j][e]) * bf16_hi(gr[e]));
      }
      *reinterpret_cast<u32x4_t *>(b + (SW_BN + r0 + 16 * j) * SK_ROWB + ch * 16) = av;
    }
  };
  // Each wave runs the whole K range on its 32 columns (two fragments, see
  // sw_col); the product is formed transposed, D[n][m] = W A^T, so a lane
  // ends with 4 consecutive columns of one row per fragment.
  f32x4_t acc[2][4];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[f][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int lr = lane & 15, lg = lane >> 4;
  auto compute = [&](int buf) {
    const uint8_t *b = sk_lds + buf * (SW_BN + SK_BM) * SK_ROWB;
#pragma unroll
    for (int ks = 0; ks < SK_KC / 32; ++ks) {
      u32x4_t wf[2], af[4];
#pragma unroll
      for (int f = 0; f < 2; ++f)
        wf[f] = *reinterpret_cast<const u32x4_t *>(b + sw_col(wave, f, lr) * SK_ROWB + (ks * 4 + lg) * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const u32x4_t *>(b + (SW_BN + i * 16 + lr) * SK_ROWB + (ks * 4 + lg) * 16);
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[f][i] = mfma16x16x32(wf[f], af[i], acc[f][i]);
    }
  };
  // Two stages in flight in registers, one in LDS: write stage s + 1 while
  // stage s is consumed, one barrier per stage.
  gload(0, wa, aa, ga);
  swrite(0, wa, aa, ga);
  gload(1, wa, aa, ga);
  gload(2, wb, ab, gb);
  __syncthreads();
  for (int st = 0; st < nst; st += 2) {
    compute(0);
    swrite(1, wa, aa, ga);
    gload(st + 3, wa, aa, ga);
    __syncthreads();
    if (st + 1 >= nst) break;
    compute(1);
    swrite(0, wb, ab, gb);
    gload(st + 4, wb, ab, gb);
    __syncthreads();
  }
  if constexpr (PRENORM) {
    // the 16 lanes of a row (chunks 0..15) hold its partial sums: one per
    // row and split (stages past nst loaded zeros and added nothing)
    if (first_col_tile) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float s = group_sum<16>(ssacc[j]);
        const int m = m0 + r0 + 16 * j;
        if (ch == 0 && m < M) ssq[(size_t)split * M + m] = s;
      }
    }
  }

  // lane: rows m = m0 + 16 i + lr; fragment f holds logical columns
  // c_f .. c_f + 3 with c_f = n0 + sw_col(wave, f, 4 lg)
  const int ncols = logical_cols(N, epi);
  int cf[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) cf[f] = n0 + sw_col(wave, f, 4 * lg);
  if constexpr (W8) {
#pragma unroll
    for (int f = 0; f < 2; ++f)
      if (cf[f] < ncols) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[f][i] = row_scaled(acc[f][i], wscale, cf[f], N, epi);
      }
  }
  if (part) {  // split-K partial, logical column space
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + i * 16 + lr;
        if (m < M && cf[f] < ncols)
          *reinterpret_cast<f32x4_t *>(part + ((size_t)split * M + m) * ncols + cf[f]) = acc[f][i];
      }
    return;
  }
  if (epi == EPI_SILU_MUL) {
    // fragment 0 holds gate sums, fragment 1 their up partners
    const int F = N >> 1;
    const int fo = ((n0 + (wave >> 1) * 64) >> 1) + (wave & 1) * 16 + 4 * lg;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i * 16 + lr;
      if (m < M && fo < F) {
        const f32x4_t g = acc[0][i], u = acc[1][i];
        const u32x2_t w = {pack_bf16x2(silu_f(g[0]) * u[0], silu_f(g[1]) * u[1]),
                           pack_bf16x2(silu_f(g[2]) * u[2], silu_f(g[3]) * u[3])};
        *reinterpret_cast<u32x2_t *>(out + (size_t)m * F + fo) = w;
      }
    }
    return;
  }
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int n = cf[f];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i * 16 + lr;
      if (m < M && n < N) {
        f32x4_t v = acc[f][i];
        if (epi == EPI_RESIDUAL) {
          const u32x2_t r = *reinterpret_cast<const u32x2_t *>(res + (size_t)m * N + n);
          v[0] += bf16_lo(r[0]);
          v[1] += bf16_hi(r[0]);
          v[2] += bf16_lo(r[1]);
          v[3] += bf16_hi(r[1]);
        }
        const u32x2_t w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        *reinterpret_cast<u32x2_t *>(out + (size_t)m * N + n) = w;
      }
    }
  }
}

// Fragment-packed weights.  A packed copy of W [N][K] (N % 16 == 0,
// K % 32 == 0) stores each 16-row x 32-column block as one contiguous
// 1 KiB run in the lane order of the MFMA's 16x16x32 operand: lane l holds
// row 16 g + l % 16, columns 32 c + 8 (l / 16) .. + 7, and block (g, c) sits
// at byte ((g * K / 32) + c) * 1024.  One 16-byte load per lane then fills an
// operand register with 1 KiB of contiguous memory.
__global__ __launch_bounds__(256) void k_pack_weight(const uint16_t *__restrict__ W, uint16_t *__restrict__ P, int N,
                                                     int K) {
  const size_t q = (size_t)blockIdx.x * 256 + threadIdx.x;  // 16-byte chunk of P
  const size_t nchunks = (size_t)N * K / 8;
  if (q >= nchunks) return;
  const int kc32 = K / 32;
  const size_t frag = q >> 6;
  const int l = (int)(q & 63);
  const size_t g = frag / kc32;
  const int c = (int)(frag - g * kc32);
  const size_t row = g * 16 + (l & 15);
  const size_t k = (size_t)c * 32 + (l >> 4) * 8;
  *reinterpret_cast<u32x4_t *>(P + q * 8) = *reinterpret_cast<const u32x4_t *>(W + row * K + k);
}

// The weight-streaming kernel on packed bf16 weights.  Same block, columns,
// split ranges, products and epilogues as k_gemm_skinny<false>, but each
// wave loads its W operands straight into registers from the packed copy
// (every element of W is used by one wave only, so W needs no LDS), three
// 128-wide K stages ahead in a ring of three register sets; only A passes
// through LDS (three buffers).  The products take the same operands in the
// same order, so the sums are bitwise those of k_gemm_skinny<false>.
constexpr int SP_LDS = 3 * SK_BM * SK_ROWB;
template <bool PRENORM = false>
__global__ __launch_bounds__(256) void k_gemm_skinny_packed(const uint16_t *__restrict__ A, const uint16_t *__restrict__ Wp,
                                                            uint16_t *__restrict__ out, const uint16_t *__restrict__ res,
                                                            float *__restrict__ part, int M, int N, int K, int epi,
                                                            int ksteps_per_split, int tiles, int mt, int per_xcd,
                                                            const uint16_t *__restrict__ gamma = nullptr,
                                                            float *__restrict__ ssq = nullptr) {
  extern __shared__ __attribute__((aligned(16))) uint8_t sp_lds[];  // [3][64 A rows][SK_ROWB]
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= tiles) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = (t / mt) * SW_BN;
  const int split = blockIdx.y;
  const int m0 = (t % mt) * SK_BM;
  const int kbeg = split * ksteps_per_split * 32;
  const int kend = min(K, kbeg + ksteps_per_split * 32);
  const int nst = kend > kbeg ? (kend - kbeg + SK_KC - 1) / SK_KC : 0;
  const buf_rsrc_t ra = make_rsrc(A, (int)min((size_t)M * K * 2, (size_t)0x7FFFFFFF));
  const buf_rsrc_t rw = make_rsrc(Wp, (int)min((size_t)N * K * 2, (size_t)0x7FFFFFFF));

  // W: fragment f of this wave covers W rows wr_f .. wr_f + 15 (a 16-aligned
  // run, or none); its 32-wide K step kc is the 1 KiB run at
  // (wr_f / 16 * K / 32 + kc) * 1024, of which this lane reads 16 bytes.
  uint32_t wbase[2];
  bool wok[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int wr = w_row_of(n0 + sw_col(wave, f, 0), N, epi);
    wok[f] = wr >= 0;
    wbase[f] = wok[f] ? ((uint32_t)(wr >> 4) * (uint32_t)(K >> 5)) * 1024u + (uint32_t)lane * 16u : 0u;
  }
  const int kc0 = kbeg >> 5, kc_end = kend >> 5;
  u32x4_t w0[2][4], w1[2][4], w2[2][4];
  auto wload = [&](int s, u32x4_t (&wr)[2][4]) {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int kc = kc0 + s * 4 + ks;
#pragma unroll
      for (int f = 0; f < 2; ++f)
        wr[f][ks] = buf_ld_u32x4<kAuxNT>(
            rw, (int)(wok[f] && s < nst && kc < kc_end ? wbase[f] + (uint32_t)kc * 1024u : 0x80000000u));
    }
  };

  // A: thread t moves 16-byte chunk t % 16 of tile rows t / 16 + 16 j (j < 4)
  const int ch = tid & 15, r0 = tid >> 4;
  uint32_t aoff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + r0 + 16 * j;
    aoff[j] = m < M ? ((uint32_t)m * (uint32_t)K + (uint32_t)(ch * 8)) * 2u : 0x80000000u;
  }
  u32x4_t aa[4];
  u32x4_t ga = {0u, 0u, 0u, 0u};
  float ssacc[4] = {0.f, 0.f, 0.f, 0.f};
  const buf_rsrc_t rg = make_rsrc(PRENORM ? gamma : A, PRENORM ? K * 2 : 16);
  auto aload = [&](int s) {
    const int k = kbeg + s * SK_KC + ch * 8;
    const bool ok = s < nst && k < kend;
    const uint32_t kb = (uint32_t)(kbeg + s * SK_KC) * 2u;
#pragma unroll
    for (int j = 0; j < 4; ++j) aa[j] = buf_ld_u32x4<0>(ra, (int)(ok ? aoff[j] + kb : 0x80000000u));
    if constexpr (PRENORM) ga = buf_ld_u32x4<0>(rg, (int)(ok ? (uint32_t)(k * 2) : 0x80000000u));
  };
  const bool first_col_tile = n0 == 0;
  auto awrite = [&](int buf) {
    uint8_t *b = sp_lds + buf * SK_BM * SK_ROWB;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x4_t av = aa[j];
      if constexpr (PRENORM) {
        if (first_col_tile) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float lo = bf16_lo(aa[j][e]), hi = bf16_hi(aa[j][e]);
            ssacc[j] += lo * lo + hi * hi;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          av[e] = bf16_pair_rne(bf16_lo(aa[j][e]) * bf16_lo(ga[e]), bf16_hi(aa[j][e]) * bf16_hi(ga[e]));
      }
      *reinterpret_cast<u32x4_t *>(b + (r0 + 16 * j) * SK_ROWB + ch * 16) = av;
    }
  };
  f32x4_t acc[2][4];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[f][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int lr = lane & 15, lg = lane >> 4;
  auto compute = [&](int buf, const u32x4_t (&wr)[2][4]) {
    const uint8_t *b = sp_lds + buf * SK_BM * SK_ROWB;
#pragma unroll
    for (int ks = 0; ks < SK_KC / 32; ++ks) {
      u32x4_t af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const u32x4_t *>(b + (i * 16 + lr) * SK_ROWB + (ks * 4 + lg) * 16);
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[f][i] = mfma16x16x32(wr[f][ks], af[i], acc[f][i]);
    }
  };
  // Stage s: compute(s) from A buffer s % 3 and W set s % 3; write A(s + 2)
  // (loaded during stage s - 1) into buffer (s + 2) % 3; load A(s + 3), then
  // W(s + 3) into the set just consumed; one barrier.  A's loads go out
  // before W's so that waiting for A(s + 2) never waits for W(s + 2).
  aload(0);
  wload(0, w0);
  awrite(0);
  aload(1);
  wload(1, w1);
  awrite(1);
  aload(2);
  wload(2, w2);
  __syncthreads();
  auto stage = [&](int s, int buf, u32x4_t (&wr)[2][4]) {
    compute(buf, wr);
    awrite(buf == 0 ? 2 : buf - 1);
    aload(s + 3);
    wload(s + 3, wr);
    __syncthreads();
  };
  int s = 0;
  for (; s + 3 <= nst; s += 3) {
    stage(s, 0, w0);
    stage(s + 1, 1, w1);
    stage(s + 2, 2, w2);
  }
  // one or two stages left: A(s) and A(s + 1) already sit in buffers 0 and 1
  if (s < nst) compute(0, w0);
  if (s + 1 < nst) compute(1, w1);
  if constexpr (PRENORM) {
    if (first_col_tile) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float v = group_sum<16>(ssacc[j]);
        const int m = m0 + r0 + 16 * j;
        if (ch == 0 && m < M) ssq[(size_t)split * M + m] = v;
      }
    }
  }

  const int ncols = logical_cols(N, epi);
  int cf[2];
#pragma unroll
  for (int f = 0; f < 2; ++f) cf[f] = n0 + sw_col(wave, f, 4 * lg);
  if (part) {
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + i * 16 + lr;
        if (m < M && cf[f] < ncols)
          *reinterpret_cast<f32x4_t *>(part + ((size_t)split * M + m) * ncols + cf[f]) = acc[f][i];
      }
    return;
  }
  if (epi == EPI_SILU_MUL) {
    const int F = N >> 1;
    const int fo = ((n0 + (wave >> 1) * 64) >> 1) + (wave & 1) * 16 + 4 * lg;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i * 16 + lr;
      if (m < M && fo < F) {
        const f32x4_t g = acc[0][i], u = acc[1][i];
        const u32x2_t w = {pack_bf16x2(silu_f(g[0]) * u[0], silu_f(g[1]) * u[1]),
                           pack_bf16x2(silu_f(g[2]) * u[2], silu_f(g[3]) * u[3])};
        *reinterpret_cast<u32x2_t *>(out + (size_t)m * F + fo) = w;
      }
    }
    return;
  }
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int n = cf[f];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + i * 16 + lr;
      if (m < M && n < N) {
        f32x4_t v = acc[f][i];
        if (epi == EPI_RESIDUAL) {
          const u32x2_t r = *reinterpret_cast<const u32x2_t *>(res + (size_t)m * N + n);
          v[0] += bf16_lo(r[0]);
          v[1] += bf16_hi(r[0]);
          v[2] += bf16_lo(r[1]);
          v[3] += bf16_hi(r[1]);
        }
        const u32x2_t w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        *reinterpret_cast<u32x2_t *>(out + (size_t)m * N + n) = w;
      }
    }
  }
}

// Sum split-K partials (logical column space) and apply the epilogue.
__global__ __launch_bounds__(256) void k_gemm_splitk_epilogue(const float *__restrict__ part, int splits,
                                                              uint16_t *__restrict__ out,
                                                              const uint16_t *__restrict__ res, int M, int N,
                                                              int epi) {
  // two consecutive output columns per thread and step (N and F are even,
  // and a SiLU group of 32 never splits a pair; two rather than four columns
  // so that a decode batch's few rows still give the chip many waves), the
  // loads of up to eight splits issued before they are added; each element
  // sums its splits in order, then adds the residual
  typedef float f2_t __attribute__((ext_vector_type(2)));
  const int ncols = logical_cols(N, epi);
  const int outc = epi == EPI_SILU_MUL ? N / 2 : N;
  const long total2 = (long)M * (outc / 2);
  const size_t stride = (size_t)M * ncols;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < total2; idx += (long)gridDim.x * blockDim.x) {
    const int m = (int)(idx / (outc / 2)), n = 2 * (int)(idx - (long)m * (outc / 2));
    const bool silu = epi == EPI_SILU_MUL;
    const int col = silu ? (n / 32) * 64 + (n & 31) : n;
    const float *p0 = part + (size_t)m * ncols + col;
    f2_t x = {0.f, 0.f}, u = {0.f, 0.f};
    for (int s0 = 0; s0 < splits; s0 += 8) {
      f2_t a[8], b[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const bool ok = s0 + q < splits;
        a[q] = ok ? *reinterpret_cast<const f2_t *>(p0 + (s0 + q) * stride) : f2_t{0.f, 0.f};
        b[q] = ok && silu ? *reinterpret_cast<const f2_t *>(p0 + (s0 + q) * stride + 32) : f2_t{0.f, 0.f};
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        x += a[q];
        u += b[q];
      }
    }
    uint32_t w;
    if (silu) {
      w = pack_bf16x2(silu_f(x[0]) * u[0], silu_f(x[1]) * u[1]);
    } else {
      if (epi == EPI_RESIDUAL) {
        const uint32_t r = *reinterpret_cast<const uint32_t *>(res + (size_t)m * N + n);
        x[0] += bf16_lo(r);
        x[1] += bf16_hi(r);
      }
      w = pack_bf16x2(x[0], x[1]);
    }
    *reinterpret_cast<uint32_t *>(out + (size_t)m * outc + n) = w;
  }
}

// ===========================================================================
// tiled
// ===========================================================================
constexpr int TL_BM = 128, TL_BN = 128, TL_BK = 64, TL_LDK = TL_BK + 8;

__global__ __launch_bounds__(256) void k_gemm_tiled(const uint16_t *__restrict__ A, const uint16_t *__restrict__ W,
                                                    uint16_t *__restrict__ out, const uint16_t *__restrict__ res,
                                                    int M, int N, int K, int epi, int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][TL_BM * TL_LDK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][TL_BN * TL_LDK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  // tile order: column-major over M inside groups of 8 N tiles, so that
  // consecutive blocks share the same A rows and a small band of W rows
  const int bid = blockIdx.x;
  const int group = 8;
  const int per_group = group * tiles_m;
  const int gidx = bid / per_group;
  const int first_n = gidx * group;
  const int gsz = min(group, tiles_n - first_n);
  const int inb = bid - gidx * per_group;
  const int tn = first_n + inb % gsz;
  const int tm = inb / gsz;
  const int m0 = tm * TL_BM, n0 = tn * TL_BN;
  const int nk = (K + TL_BK - 1) / TL_BK;

  // global -> register staging: 4 chunks of 16 B for A and for W per thread
  const int ldr = threadIdx.x >> 3;        // row 0..31 within a pass
  const int ldc = (threadIdx.x & 7) * 8;   // k offset
  const uint16_t *ga[4];
  const uint16_t *gb[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int m = m0 + p * 32 + ldr;
    ga[p] = m < M ? A + (size_t)m * K : nullptr;
    const int wr = w_row_of(n0 + p * 32 + ldr, N, epi);
    gb[p] = wr >= 0 ? W + (size_t)wr * K : nullptr;
  }
  u32x4_t ra[4], rb[4];
  auto gload = [&](int kt) {
    const int k = kt * TL_BK + ldc;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      ra[p] = (ga[p] && k < K) ? ld_u32x4(ga[p] + k) : u32x4_t{0, 0, 0, 0};
      rb[p] = (gb[p] && k < K) ? ld_u32x4(gb[p] + k) : u32x4_t{0, 0, 0, 0};
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      st_u32x4(&sA[buf][(p * 32 + ldr) * TL_LDK + ldc], ra[p]);
      st_u32x4(&sB[buf][(p * 32 + ldr) * TL_LDK + ldc], rb[p]);
    }
  };
  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lk = (lane >> 4) * 8;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < TL_BK; kk += 32) {
      u32x4_t a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = ld_u32x4(&sA[buf][(wm * 64 + i * 16 + lr) * TL_LDK + kk + lk]);
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = ld_u32x4(&sB[buf][(wn * 64 + j * 16 + lr) * TL_LDK + kk + lk]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }
  // epilogue straight from the accumulator layout: lane holds rows
  // 4 (lane/16) + e, column lane % 16 of each 16x16 block
  const int cbase = n0 + wn * 64;
  if (epi == EPI_SILU_MUL) {
    const int F = N >> 1;
    const int f0 = cbase >> 1;  // 64-group -> 32 ffn columns
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + e;
          const int f = f0 + j * 16 + lr;
          if (m < M && f < F)
            out[(size_t)m * F + f] = (uint16_t)f32_to_bf16_bits(silu_f(acc[i][j][e]) * acc[i][j + 2][e]);
        }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + e;
        const int n = cbase + j * 16 + lr;
        if (m < M && n < N) {
          float x = acc[i][j][e];
          if (epi == EPI_RESIDUAL) x += bf16_to_f32(res[(size_t)m * N + n]);
          out[(size_t)m * N + n] = (uint16_t)f32_to_bf16_bits(x);
        }
      }
}

// ===========================================================================
// big: 256 x 256 output tiles for large M (prefill-sized batches).  K tiles
// of 64 stream into a double-buffered LDS ring straight from global memory
// (buffer loads with an LDS destination: no register round trip).  8 waves
// (2 along M x 4 along N) each own a 128 x 64 sub-tile held in accumulation
// registers.  The product is formed transposed, C^T = W A^T, so that each
// lane's accumulators hold 4 consecutive output columns of one row and the
// epilogue stores 8 bytes at a time.  LDS rows are 128 bytes (64 bf16 of
// K); the 16-byte chunk c of row r sits at chunk c ^ ((r >> 1) & 7), which
// makes the MFMA operand reads of 16 consecutive rows conflict free.
// With fewer tiles than CUs (decode-sized M of 256 against a few thousand
// columns) blocks split K (gridDim.y splits of kt_per K tiles) and write
// fp32 partials in logical column space for the split-K epilogue kernel.
// Requires K % 64 == 0, N % 8 == 0 and both operands under 2 GiB (32-bit
// offsets).
// ===========================================================================
constexpr int BG_BM = 256, BG_BN = 256, BG_BK = 64;
constexpr int BG_THREADS = 512;
constexpr int BG_TILE_BYTES = 256 * BG_BK * 2;  // one operand tile: 32 KiB

__device__ __forceinline__ int bg_swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Grouped use (the experts of a mixture-of-experts block): a tile is up to
// 256 expert-sorted rows of one expert (tables [3][max_tiles]: expert, first
// sorted row, rows); block b takes tile b / tiles_n and column tile
// b % tiles_n of that expert's W ([E][N][K]); A rows are gathered through
// a_rows (null: the sorted row itself); the store epilogue may write fp32.
struct GroupedArgs {
  const int32_t *a_rows, *tiles, *n_tiles;
  int max_tiles, a_nrows, f32_out;
};

template <bool W8, bool GROUPED>
__global__ __launch_bounds__(BG_THREADS) void k_gemm_big(const uint16_t *__restrict__ A, const void *__restrict__ W,
                                                         const float *__restrict__ wscale, uint16_t *__restrict__ out,
                                                         const uint16_t *__restrict__ res, float *__restrict__ part,
                                                         int M, int N, int K, int epi, int tiles_m, int tiles_n,
                                                         int per_xcd, int kt_per, GroupedArgs ga) {
  extern __shared__ __attribute__((aligned(16))) uint8_t bg_lds[];  // [2][A tile | W tile]
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 2, wn = wave & 3;  // 128 rows of M, 64 columns of N
  // XCD-aware tile order: blocks are dealt round-robin to the 8 XCDs, so
  // block b works on tile (b % 8) * per_xcd + b / 8: each XCD walks its own
  // contiguous run of the (grouped) tile order and its L2 keeps the shared
  // A and W panels.
  int m0, n0, mlim;  // first row, first logical column, rows of the tile in use
  const void *Wt = W;
  if constexpr (GROUPED) {
    const int rt = blockIdx.x / tiles_n;
    if (rt >= __builtin_amdgcn_readfirstlane(*ga.n_tiles)) return;
    const int e = __builtin_amdgcn_readfirstlane(ga.tiles[rt]);
    m0 = __builtin_amdgcn_readfirstlane(ga.tiles[ga.max_tiles + rt]);
    mlim = __builtin_amdgcn_readfirstlane(ga.tiles[2 * ga.max_tiles + rt]);
    n0 = (blockIdx.x % tiles_n) * BG_BN;
    Wt = static_cast<const uint16_t *>(W) + (size_t)e * N * K;
  } else {
    const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (t >= tiles_m * tiles_n) return;
    const int group = 8;
    const int per_group = group * tiles_m;
    const int gidx = t / per_group;
    const int first_n = gidx * group;
    const int gsz = min(group, tiles_n - first_n);
    const int inb = t - gidx * per_group;
    const int tn = first_n + inb % gsz;
    const int tm = inb / gsz;
    m0 = tm * BG_BM;
    n0 = tn * BG_BN;
    mlim = M - m0;
  }
  const int split = blockIdx.y;
  const int kt0 = split * kt_per, kt1 = min(K / BG_BK, kt0 + kt_per);

  constexpr uint32_t WES = W8 ? 1u : 2u;  // bytes per W element
  const int a_nrows = GROUPED ? ga.a_nrows : M;
  const buf_rsrc_t ra = make_rsrc(A, (int)min((size_t)a_nrows * K * 2, (size_t)0x7FFFFFFF));
  const buf_rsrc_t rw = make_rsrc(Wt, (int)min((size_t)N * K * WES, (size_t)0x7FFFFFFF));
  // DMA: wave w moves LDS rows [32 w, 32 w + 32) of both tiles, 8 rows
  // (1 KiB) per instruction; lane l fills row 8 i + l / 8, physical chunk
  // l % 8 with logical chunk bg_swz(row, l % 8).  Rows outside the operands
  // point 2 GiB in, past every descriptor's range, so they load zeros.
  uint32_t aoff[4], woff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wave * 32 + i * 8 + (lane >> 3);
    const int c = bg_swz(row, lane & 7);
    int ar = row < mlim ? m0 + row : -1;
    if constexpr (GROUPED)
      if (ar >= 0 && ga.a_rows) ar = ga.a_rows[ar];
    aoff[i] = ar >= 0 && ar < a_nrows ? ((uint32_t)ar * (uint32_t)K + (uint32_t)(c * 8)) * 2u : 0x80000000u;
    const int wr = w_row_of(n0 + row, N, epi);
    woff[i] = wr >= 0 ? ((uint32_t)wr * (uint32_t)K + (uint32_t)(c * 8)) * WES : 0x80000000u;
  }
  typedef __attribute__((address_space(3))) void lds_void;
  // 8-bit weights come through registers: lane l of wave w holds the 8
  // codes of row 32 w + 8 i + l / 8, logical chunk bg_swz(row, l % 8) (the
  // same positions the DMA fills), converted to bf16 when written to LDS
  u32x2_t wcodes[4];
  auto dma = [&](int kt, int buf) {
    uint8_t *base = bg_lds + buf * 2 * BG_TILE_BYTES + wave * 32 * 128;
    const uint32_t kb = (uint32_t)kt * BG_BK * 2u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(base + i * 1024), 16, aoff[i] + kb, 0, 0, 0);
      if constexpr (W8)
        wcodes[i] = buf_ld_u32x2<0>(rw, (int)(woff[i] == 0x80000000u ? woff[i] : woff[i] + kb / 2u));
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void *)(base + BG_TILE_BYTES + i * 1024), 16, woff[i] + kb,
                                                 0, 0, 0);
    }
  };
  auto wstore = [&](int buf) {  // 8-bit weights: the converted W tile of the last dma into LDS
    uint8_t *base = bg_lds + buf * 2 * BG_TILE_BYTES + BG_TILE_BYTES + wave * 32 * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<u32x4_t *>(base + i * 1024 + lane * 16) = e4m3x8_to_bf16x8(wcodes[i]);
  };

  f32x4_t acc[4][8];  // [W block jn][A block im]: rows n, cols m
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lg = lane >> 4;
  dma(kt0, 0);
  if constexpr (W8) wstore(0);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    if (kt + 1 < kt1) dma(kt + 1, buf ^ 1);
    const uint8_t *sa = bg_lds + buf * 2 * BG_TILE_BYTES;
    const uint8_t *sw = sa + BG_TILE_BYTES;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      u32x4_t af[8], wf[4];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = wm * 128 + i * 16 + lr;
        af[i] = *reinterpret_cast<const u32x4_t *>(sa + r * 128 + bg_swz(r, ks * 4 + lg) * 16);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = wn * 64 + j * 16 + lr;
        wf[j] = *reinterpret_cast<const u32x4_t *>(sw + r * 128 + bg_swz(r, ks * 4 + lg) * 16);
      }
#pragma unroll
      for (int jn = 0; jn < 4; ++jn)
#pragma unroll
        for (int im = 0; im < 8; ++im) acc[jn][im] = mfma16x16x32(wf[jn], af[im], acc[jn][im]);
    }
    // the other buffer was last read in the previous step, before its barrier
    if constexpr (W8)
      if (kt + 1 < kt1) wstore(buf ^ 1);
    __syncthreads();
  }
  if constexpr (W8) {  // the rows' scales, before any epilogue or partial
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      const int n = n0 + wn * 64 + jn * 16 + lg * 4;
      if (n < logical_cols(N, epi)) {
#pragma unroll
        for (int im = 0; im < 8; ++im) acc[jn][im] = row_scaled(acc[jn][im], wscale, n, N, epi);
      }
    }
  }

  // epilogue: lane holds out[m][n .. n+3] with m = m0 + wm*128 + 16 im + lr,
  // n = n0 + wn*64 + 16 jn + 4 lg (N and F are multiples of 4, so a group of
  // 4 columns is either wholly inside or wholly outside)
  if (part) {  // split-K partial, logical column space
    const int ncols = logical_cols(N, epi);
#pragma unroll
    for (int jn = 0; jn < 4; ++jn) {
      const int n = n0 + wn * 64 + jn * 16 + lg * 4;
#pragma unroll
      for (int im = 0; im < 8; ++im) {
        const int m = m0 + wm * 128 + im * 16 + lr;
        if (m - m0 < mlim && n < ncols) *reinterpret_cast<f32x4_t *>(part + ((size_t)split * M + m) * ncols + n) = acc[jn][im];
      }
    }
    return;
  }
  if (epi == EPI_SILU_MUL) {
    // the wave's 64 columns are one [32 gate | 32 up] group: blocks jn and
    // jn + 2 pair up
    const int F = N >> 1;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int f = ((n0 + wn * 64) >> 1) + jj * 16 + lg * 4;
#pragma unroll
      for (int im = 0; im < 8; ++im) {
        const int m = m0 + wm * 128 + im * 16 + lr;
        if (m - m0 < mlim && f < F) {
          const f32x4_t gv = acc[jj][im], uv = acc[jj + 2][im];
          u32x2_t w = {pack_bf16x2(silu_f(gv[0]) * uv[0], silu_f(gv[1]) * uv[1]),
                       pack_bf16x2(silu_f(gv[2]) * uv[2], silu_f(gv[3]) * uv[3])};
          *reinterpret_cast<u32x2_t *>(out + (size_t)m * F + f) = w;
        }
      }
    }
    return;
  }
#pragma unroll
  for (int jn = 0; jn < 4; ++jn) {
    const int n = n0 + wn * 64 + jn * 16 + lg * 4;
#pragma unroll
    for (int im = 0; im < 8; ++im) {
      const int m = m0 + wm * 128 + im * 16 + lr;
      if (m - m0 < mlim && n < N) {
        f32x4_t v = acc[jn][im];
        if constexpr (GROUPED) {
          if (ga.f32_out) {
            *reinterpret_cast<f32x4_t *>(reinterpret_cast<float *>(out) + (size_t)m * N + n) = v;
            continue;
          }
        }
        if (epi == EPI_RESIDUAL) {
          const u32x2_t r = *reinterpret_cast<const u32x2_t *>(res + (size_t)m * N + n);
          v[0] += bf16_lo(r[0]);
          v[1] += bf16_hi(r[0]);
          v[2] += bf16_lo(r[1]);
          v[3] += bf16_hi(r[1]);
        }
        u32x2_t w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        *reinterpret_cast<u32x2_t *>(out + (size_t)m * N + n) = w;
      }
    }
  }
}

// ===========================================================================
// grouped: the experts of a mixture-of-experts block
// ===========================================================================
// Rows are sorted by expert; a row tile is up to 64 consecutive sorted rows of
// one expert (tile tables: expert, first sorted row, rows).  Block b takes row
// tile b / col_tiles and column tile b % col_tiles of that expert's W, so the
// column tiles of one row tile run side by side and share its A rows, and
// the row tiles of one expert follow each other and share its W tiles in L2.
// The main loop stages W and A through LDS in 128-wide K slices as the
// weight-streaming kernel does; here the 4 waves split the tile's 64 columns
// (16 each, transposed product).  A rows are gathered through a_rows (null: the sorted row
// itself).  SiLU: bf16 [rows, N / 2]; store: fp32 [rows, N].
template <bool F32OUT>
__global__ __launch_bounds__(256) void k_gemm_grouped(const uint16_t *__restrict__ A, int a_nrows,
                                                      const int32_t *__restrict__ a_rows,
                                                      const uint16_t *__restrict__ W, void *__restrict__ out,
                                                      const int32_t *__restrict__ tiles,
                                                      const int32_t *__restrict__ n_tiles, int max_tiles, int N,
                                                      int K, int epi, int col_tiles) {
  extern __shared__ __attribute__((aligned(16))) uint8_t gg_lds[];  // [2][64 W rows + 64 A rows][SK_ROWB]
  const int rt = blockIdx.x / col_tiles, ct = blockIdx.x % col_tiles;
  if (rt >= __builtin_amdgcn_readfirstlane(*n_tiles)) return;
  const int e = __builtin_amdgcn_readfirstlane(tiles[rt]);
  const int row0 = __builtin_amdgcn_readfirstlane(tiles[max_tiles + rt]);
  const int rows = __builtin_amdgcn_readfirstlane(tiles[2 * max_tiles + rt]);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = ct * SK_BN;
  const int nst = (K + SK_KC - 1) / SK_KC;
  const uint16_t *We = W + (size_t)e * N * K;
  const buf_rsrc_t ra = make_rsrc(A, (int)min((size_t)a_nrows * K * 2, (size_t)0x7FFFFFFF));
  const buf_rsrc_t rw = make_rsrc(We, (int)min((size_t)N * K * 2, (size_t)0x7FFFFFFF));

  // staging as in the weight-streaming kernel: thread t moves 16-byte chunk
  // t % 16 of tile rows t / 16 + 16 j; rows outside the tile or the operands
  // and k past K load zeros without memory traffic
  const int ch = tid & 15, r0 = tid >> 4;
  uint32_t woff[4], aoff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int wr = w_row_of(n0 + r0 + 16 * j, N, epi);
    woff[j] = wr >= 0 ? ((uint32_t)wr * (uint32_t)K + (uint32_t)(ch * 8)) * 2u : 0x80000000u;
    const int r = r0 + 16 * j;
    const int ar = r < rows ? (a_rows ? a_rows[row0 + r] : row0 + r) : -1;
    aoff[j] = ar >= 0 && ar < a_nrows ? ((uint32_t)ar * (uint32_t)K + (uint32_t)(ch * 8)) * 2u : 0x80000000u;
  }
  u32x4_t wa[4], aa[4], wb[4], ab[4];
  auto gload = [&](int s, u32x4_t (&wr)[4], u32x4_t (&ar)[4]) {
    const int k = s * SK_KC + ch * 8;
    const bool ok = s < nst && k < K;
    const uint32_t kb = (uint32_t)(s * SK_KC) * 2u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      wr[j] = buf_ld_u32x4<kAuxNT>(rw, (int)(ok ? woff[j] + kb : 0x80000000u));
      ar[j] = buf_ld_u32x4<0>(ra, (int)(ok ? aoff[j] + kb : 0x80000000u));
    }
  };
  auto swrite = [&](int buf, const u32x4_t (&wr)[4], const u32x4_t (&ar)[4]) {
    uint8_t *b = gg_lds + buf * (SK_BN + SK_BM) * SK_ROWB;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *reinterpret_cast<u32x4_t *>(b + (r0 + 16 * j) * SK_ROWB + ch * 16) = wr[j];
      *reinterpret_cast<u32x4_t *>(b + (SK_BN + r0 + 16 * j) * SK_ROWB + ch * 16) = ar[j];
    }
  };
  f32x4_t acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int lr = lane & 15, lg = lane >> 4;
  const int my_wrow = sk_col(wave, lr);
  auto compute = [&](int buf) {
    const uint8_t *b = gg_lds + buf * (SK_BN + SK_BM) * SK_ROWB;
#pragma unroll
    for (int ks = 0; ks < SK_KC / 32; ++ks) {
      const u32x4_t wf = *reinterpret_cast<const u32x4_t *>(b + my_wrow * SK_ROWB + (ks * 4 + lg) * 16);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const u32x4_t af = *reinterpret_cast<const u32x4_t *>(b + (SK_BN + i * 16 + lr) * SK_ROWB + (ks * 4 + lg) * 16);
        acc[i] = mfma16x16x32(wf, af, acc[i]);
      }
    }
  };
  gload(0, wa, aa);
  swrite(0, wa, aa);
  gload(1, wa, aa);
  gload(2, wb, ab);
  __syncthreads();
  for (int st = 0; st < nst; st += 2) {
    compute(0);
    swrite(1, wa, aa);
    gload(st + 3, wa, aa);
    __syncthreads();
    if (st + 1 >= nst) break;
    compute(1);
    swrite(0, wb, ab);
    gload(st + 4, wb, ab);
    __syncthreads();
  }

  // lane: tile rows 16 i + lr, logical columns c .. c + 3, c = sk_col(wave, 4 lg)
  const int c = sk_col(wave, 4 * lg);
  if (epi == EPI_SILU_MUL) {
    const int F = N >> 1;
    const int f = (n0 >> 1) + 8 * wave + 4 * lg;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4_t u;
#pragma unroll
      for (int q = 0; q < 4; ++q) u[q] = shfl_xor_f32(acc[i][q], 32);
      const int m = i * 16 + lr;
      if (!F32OUT && lg < 2 && m < rows && f < F) {
        const u32x2_t w = {pack_bf16x2(silu_f(acc[i][0]) * u[0], silu_f(acc[i][1]) * u[1]),
                           pack_bf16x2(silu_f(acc[i][2]) * u[2], silu_f(acc[i][3]) * u[3])};
        *reinterpret_cast<u32x2_t *>(static_cast<uint16_t *>(out) + (size_t)(row0 + m) * F + f) = w;
      }
    }
    return;
  }
  const int n = n0 + c;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = i * 16 + lr;
    if (m < rows && n < N) {
      if constexpr (F32OUT)
        *reinterpret_cast<f32x4_t *>(static_cast<float *>(out) + (size_t)(row0 + m) * N + n) = acc[i];
      else
        *reinterpret_cast<u32x2_t *>(static_cast<uint16_t *>(out) + (size_t)(row0 + m) * N + n) =
            u32x2_t{pack_bf16x2(acc[i][0], acc[i][1]), pack_bf16x2(acc[i][2], acc[i][3])};
    }
  }
}

// ===========================================================================
// planning and launch
// ===========================================================================
// Row counts up to this use the skinny kernel (weight streaming: the row
// blocks of a column tile run side by side and read W once from HBM).
constexpr int kSkinnyMaxRows = 256;

// The split-K sum of a residual GEMM and the RMSNorm of its rows in one
// pass: h = bf16(sum_s part[s] + res) is stored (the splits summed in order,
// as the split-K epilogue does), then out = bf16(h * inv * g) with inv from
// the rounded h.  One block of kFuseThreads per row (a decode batch has few
// rows, so the row's loads are spread over many waves): thread t takes the
// 8-column chunks t, t + kFuseThreads, .. (rows up to kFuseThreads *
// kFuseMaxChunks chunks wide), issues the loads of eight splits before
// adding them, and the sum of squares is reduced across the block.
constexpr int kFuseThreads = 512;
constexpr int kFuseMaxChunks = 2;
__global__ __launch_bounds__(kFuseThreads) void k_splitk_residual_rmsnorm(const float *__restrict__ part, int splits,
                                                                 const uint16_t *__restrict__ res,
                                                                 uint16_t *__restrict__ h,
                                                                 const uint16_t *__restrict__ g,
                                                                 uint16_t *__restrict__ out, int M, int N,
                                                                 float eps) {
  __shared__ float red[kFuseThreads / 64];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  const int nch = N >> 3;
  u32x4_t v[kFuseMaxChunks];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kFuseMaxChunks; ++j) {
    const int c = tid + kFuseThreads * j;
    v[j] = u32x4_t{0u, 0u, 0u, 0u};
    if (c < nch) {
      f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
      const float *pp = part + (size_t)row * N + c * 8;
      const size_t stride = (size_t)M * N;
      for (int s0i = 0; s0i < splits; s0i += 8) {
        f32x4_t a[8], b[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const bool ok = s0i + q < splits;
          a[q] = ok ? *reinterpret_cast<const f32x4_t *>(pp + (s0i + q) * stride) : f32x4_t{0.f, 0.f, 0.f, 0.f};
          b[q] = ok ? *reinterpret_cast<const f32x4_t *>(pp + (s0i + q) * stride + 4) : f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          s0 += a[q];
          s1 += b[q];
        }
      }
      const u32x4_t r = ld_u32x4(res + (size_t)row * N + c * 8);
      s0[0] += bf16_lo(r[0]);
      s0[1] += bf16_hi(r[0]);
      s0[2] += bf16_lo(r[1]);
      s0[3] += bf16_hi(r[1]);
      s1[0] += bf16_lo(r[2]);
      s1[1] += bf16_hi(r[2]);
      s1[2] += bf16_lo(r[3]);
      s1[3] += bf16_hi(r[3]);
      v[j] = u32x4_t{pack_bf16x2(s0[0], s0[1]), pack_bf16x2(s0[2], s0[3]), pack_bf16x2(s1[0], s1[1]),
                     pack_bf16x2(s1[2], s1[3])};
      st_u32x4(h + (size_t)row * N + c * 8, v[j]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = bf16_lo(v[j][i]), y = bf16_hi(v[j][i]);
        ss += x * x + y * y;
      }
    }
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kFuseThreads / 64; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)N + eps);
#pragma unroll
  for (int j = 0; j < kFuseMaxChunks; ++j) {
    const int c = tid + kFuseThreads * j;
    if (c < nch) {
      const u32x4_t gv = ld_u32x4(g + c * 8);
      u32x4_t o;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        o[i] = pack_bf16x2(bf16_lo(v[j][i]) * inv * bf16_lo(gv[i]), bf16_hi(v[j][i]) * inv * bf16_hi(gv[i]));
      st_u32x4(out + (size_t)row * N + c * 8, o);
    }
  }
}

// The split-K sum and epilogue, or with nf (residual epilogue, rows fit) the
// sum fused with the RMSNorm of the result rows (nf->done set).
static hipError_t finish_splitk(const float *part, int splits, uint16_t *out, const uint16_t *res, int M, int N,
                                int epi, NormFuse *nf, hipStream_t st);

static hipError_t launch_splitk_epilogue(const float *part, int splits, uint16_t *out, const uint16_t *res, int M,
                                         int N, int epi, hipStream_t st) {
  const int outc = epi == EPI_SILU_MUL ? N / 2 : N;
  const long total = (long)M * (outc / 2);
  const int blocks = (int)((total + 255) / 256 < 8192 ? (total + 255) / 256 : 8192);
  hipLaunchKernelGGL(k_gemm_splitk_epilogue, dim3(blocks), dim3(256), 0, st, part, splits, out, res, M, N, epi);
  return hipGetLastError();
}

static hipError_t finish_splitk(const float *part, int splits, uint16_t *out, const uint16_t *res, int M, int N,
                                int epi, NormFuse *nf, hipStream_t st) {
  if (nf && nf->gamma && epi == EPI_RESIDUAL && N % 8 == 0 && N / 8 <= kFuseThreads * kFuseMaxChunks) {
    hipLaunchKernelGGL(k_splitk_residual_rmsnorm, dim3(M), dim3(kFuseThreads), 0, st, part, splits, res, out, nf->gamma,
                       nf->out, M, N, nf->eps);
    nf->done = true;
    return hipGetLastError();
  }
  return launch_splitk_epilogue(part, splits, out, res, M, N, epi, st);
}

static int skinny_splits(int M, int N, int K) {
  const int tiles = ((N + SW_BN - 1) / SW_BN) * ((M + SK_BM - 1) / SK_BM);
  const int nsteps = (K + 31) / 32;
  // one block per CU (256 CUs).  A grid that covers at least 3/4 of the CUs
  // is not split; otherwise K is split into the count whose rounds of 256
  // blocks take the least time per split (ceil(tiles s / 256) / s; fewer
  // splits on ties), at most 8 (the fp32 partials are written and read back
  // once per split) and each split keeping 4 or more 128-wide K stages
  if (tiles >= 192) return 1;
  int best = 1;
  for (int s = 2; s <= 8 && nsteps / s >= 16; ++s) {
    const long rs = ((long)tiles * s + 255) / 256, rb = ((long)tiles * best + 255) / 256;
    if (rs * best < rb * s) best = s;  // rs / s < rb / best
  }
  return best;
}

GemmPlan plan_gemm(int M, int N, int K, int epi, bool w8) {
  GemmPlan p{};
  p.splits = 1;
  if (M <= 0 || N <= 0 || K <= 0) return p;  // nothing to plan (kind 0, no workspace)
  const int ncols = logical_cols(N, epi);
  // the big kernel addresses W through a 32-bit buffer range; A is cut into
  // row chunks that each fit one (launch_gemm)
  const bool fits = (size_t)N * K * 2 < ((size_t)1 << 31) && (size_t)BG_BM * K * 2 < ((size_t)1 << 31);
  // 256 x 256 tiles once the grid covers at least half the CUs
  const long big_tiles = (long)((M + BG_BM - 1) / BG_BM) * ((ncols + BG_BN - 1) / BG_BN);
  if (K % BG_BK == 0 && N % 8 == 0 && fits && M >= 256) {
    // one block per CU: split K while the tiles cover at most half the CUs,
    // keeping at least 8 K tiles per split
    p.kind = 2;
    const int nk = K / BG_BK;
    int splits = 1;
    if (big_tiles <= 128 && (size_t)M * K * 2 < ((size_t)1 << 31)) {
      const long by_cus = 256 / big_tiles, by_k = nk / 8;
      splits = (int)(by_cus < by_k ? by_cus : by_k);
    }
    if (splits < 1) splits = 1;
    p.kt_per = (nk + splits - 1) / splits;
    p.splits = (nk + p.kt_per - 1) / p.kt_per;
    p.ws_bytes = p.splits > 1 ? (size_t)p.splits * M * ncols * sizeof(float) : 0;
    return p;
  }
  // the skinny kernel addresses both operands through 32-bit buffer ranges
  const bool sk_fits = (size_t)N * K * (w8 ? 1 : 2) < ((size_t)1 << 31) && (size_t)M * K * 2 < ((size_t)1 << 31);
  if ((M <= kSkinnyMaxRows || w8) && sk_fits) {  // (the tiled kernel reads bf16 weights only)
    p.kind = 0;
    p.splits = skinny_splits(M, ncols, K);
    p.ws_bytes = p.splits > 1 ? (size_t)p.splits * M * ncols * sizeof(float) : 0;
    return p;
  }
  p.kind = w8 ? -1 : 1;  // -1: no kernel here addresses 8-bit operands this large
  p.splits = 1;
  p.ws_bytes = 0;
  return p;
}

bool packed_ok(int N, int K, int epi) {
  if (N <= 0 || K <= 0 || N % 16 || K % 32) return false;
  if (epi == EPI_SILU_MUL && (N / 2) % 16) return false;  // gate and up runs must stay 16-aligned
  return (size_t)N * K * 2 < ((size_t)1 << 31);
}

size_t packed_weight_bytes(int N, int K) { return (size_t)N * K * 2; }

hipError_t pack_weight(const uint16_t *W, uint16_t *P, int N, int K, hipStream_t st) {
  if (!W || !P || N <= 0 || K <= 0 || N % 16 || K % 32) return hipErrorInvalidValue;
  const size_t chunks = (size_t)N * K / 8;
  const size_t blocks = (chunks + 255) / 256;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_pack_weight, dim3((unsigned)blocks), dim3(256), 0, st, W, P, N, K);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmPlan &p, const uint16_t *A, const void *W, const float *wscale, uint16_t *out,
                       const uint16_t *res, int M, int N, int K, int epi, void *ws, hipStream_t st, NormFuse *nf,
                       const uint16_t *Wp) {
  if (nf) nf->done = false;
  if (M <= 0) return hipSuccess;
  const bool w8 = wscale != nullptr;
  if (p.kind < 0 || (w8 && p.kind == 1)) return hipErrorInvalidValue;
  const int ncols = logical_cols(N, epi);
  if (p.kind == 0) {
    const int nsteps = (K + 31) / 32;
    const int splits = p.splits;
    const int per = (nsteps + splits - 1) / splits;
    float *part = splits > 1 ? reinterpret_cast<float *>(ws) : nullptr;
    const int mt = (M + SK_BM - 1) / SK_BM;
    const int tiles = ((ncols + SW_BN - 1) / SW_BN) * mt;
    const int per_xcd = (tiles + 7) / 8;
    dim3 grid(8 * per_xcd, splits);
    if (w8)
      hipLaunchKernelGGL(k_gemm_skinny<true>, grid, dim3(256), SW_LDS, st, A, W, wscale, out, res, part, M, N, K, epi,
                         per, tiles, mt, per_xcd);
    else if (Wp && packed_ok(N, K, epi))  // (SW_LDS of LDS keeps one block per CU)
      hipLaunchKernelGGL(k_gemm_skinny_packed<false>, grid, dim3(256), SW_LDS, st, A, Wp, out, res, part, M, N, K,
                         epi, per, tiles, mt, per_xcd);
    else
      hipLaunchKernelGGL(k_gemm_skinny<false>, grid, dim3(256), SW_LDS, st, A, W, wscale, out, res, part, M, N, K,
                         epi, per, tiles, mt, per_xcd);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1) return e;
    return finish_splitk(part, splits, out, res, M, N, epi, nf, st);
  }
  if (p.kind == 2) {
    if (p.splits > 1) {  // one launch (the plan only splits a few tiles), then the partial sums
      const int tm = (M + BG_BM - 1) / BG_BM, tn = (ncols + BG_BN - 1) / BG_BN;
      const int per_xcd = (tm * tn + 7) / 8;
      float *part = reinterpret_cast<float *>(ws);
      if (w8)
        hipLaunchKernelGGL((k_gemm_big<true, false>), dim3(8 * per_xcd, p.splits), dim3(BG_THREADS), 4 * BG_TILE_BYTES, st, A,
                           W, wscale, out, res, part, M, N, K, epi, tm, tn, per_xcd, p.kt_per, GroupedArgs{});
      else
        hipLaunchKernelGGL((k_gemm_big<false, false>), dim3(8 * per_xcd, p.splits), dim3(BG_THREADS), 4 * BG_TILE_BYTES, st, A,
                           W, wscale, out, res, part, M, N, K, epi, tm, tn, per_xcd, p.kt_per, GroupedArgs{});
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      return finish_splitk(part, p.splits, out, res, M, N, epi, nf, st);
    }
    // rows per launch: A's slice must stay inside a 32-bit buffer range
    const size_t rows_fit = ((((size_t)1 << 31) - 1) / ((size_t)K * 2)) / BG_BM * BG_BM;
    const int chunk = (int)(rows_fit < (size_t)M ? rows_fit : (size_t)M);
    const size_t out_cols = epi == EPI_SILU_MUL ? (size_t)N / 2 : (size_t)N;
    for (int m0 = 0; m0 < M; m0 += chunk) {
      const int mc = M - m0 < chunk ? M - m0 : chunk;
      const int tm = (mc + BG_BM - 1) / BG_BM, tn = (ncols + BG_BN - 1) / BG_BN;
      const int per_xcd = (tm * tn + 7) / 8;
      if (w8)
        hipLaunchKernelGGL((k_gemm_big<true, false>), dim3(8 * per_xcd), dim3(BG_THREADS), 4 * BG_TILE_BYTES, st,
                           A + (size_t)m0 * K, W, wscale, out + (size_t)m0 * out_cols,
                           res ? res + (size_t)m0 * N : nullptr, nullptr, mc, N, K, epi, tm, tn, per_xcd, K / BG_BK,
                           GroupedArgs{});
      else
        hipLaunchKernelGGL((k_gemm_big<false, false>), dim3(8 * per_xcd), dim3(BG_THREADS), 4 * BG_TILE_BYTES, st,
                           A + (size_t)m0 * K, W, wscale, out + (size_t)m0 * out_cols,
                           res ? res + (size_t)m0 * N : nullptr, nullptr, mc, N, K, epi, tm, tn, per_xcd, K / BG_BK,
                           GroupedArgs{});
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const int tiles_m = (M + TL_BM - 1) / TL_BM, tiles_n = (ncols + TL_BN - 1) / TL_BN;
  hipLaunchKernelGGL(k_gemm_tiled, dim3(tiles_m * tiles_n), dim3(256), 0, st, A,
                     static_cast<const uint16_t *>(W), out, res, M, N, K, epi, tiles_m,
                     tiles_n);
  return hipGetLastError();
}

hipError_t launch_gemm_prenorm(const GemmPlan &p, const uint16_t *x, const uint16_t *gamma, const void *W,
                               const float *wscale, int M, int N, int K, float *part, float *ssq, hipStream_t st,
                               const uint16_t *Wp) {
  if (M <= 0) return hipSuccess;
  if (p.kind != 0 || p.splits < 2) return hipErrorInvalidValue;
  const int nsteps = (K + 31) / 32;
  const int per = (nsteps + p.splits - 1) / p.splits;
  const int mt = (M + SK_BM - 1) / SK_BM;
  const int tiles = ((N + SW_BN - 1) / SW_BN) * mt;
  const int per_xcd = (tiles + 7) / 8;
  dim3 grid(8 * per_xcd, p.splits);
  if (wscale)
    hipLaunchKernelGGL((k_gemm_skinny<true, true>), grid, dim3(256), SW_LDS, st, x, W, wscale, nullptr, nullptr, part,
                       M, N, K, (int)EPI_STORE, per, tiles, mt, per_xcd, gamma, ssq);
  else if (Wp && packed_ok(N, K, EPI_STORE))
    hipLaunchKernelGGL((k_gemm_skinny_packed<true>), grid, dim3(256), SW_LDS, st, x, Wp, nullptr, nullptr, part, M, N,
                       K, (int)EPI_STORE, per, tiles, mt, per_xcd, gamma, ssq);
  else
    hipLaunchKernelGGL((k_gemm_skinny<false, true>), grid, dim3(256), SW_LDS, st, x, W, wscale, nullptr, nullptr,
                       part, M, N, K, (int)EPI_STORE, per, tiles, mt, per_xcd, gamma, ssq);
  return hipGetLastError();
}

hipError_t launch_gemm_grouped_big(const uint16_t *A, int a_nrows, const int32_t *a_rows, const uint16_t *W,
                                   void *out, bool f32_out, const int32_t *tiles, const int32_t *n_tiles, int max_tiles,
                                   int N, int K, int epi, hipStream_t st) {
  if (max_tiles <= 0) return hipSuccess;
  if (K % BG_BK) return hipErrorInvalidValue;
  const int tiles_n = (logical_cols(N, epi) + BG_BN - 1) / BG_BN;
  const GroupedArgs ga{a_rows, tiles, n_tiles, max_tiles, a_nrows, f32_out ? 1 : 0};
  hipLaunchKernelGGL((k_gemm_big<false, true>), dim3((unsigned)max_tiles * (unsigned)tiles_n), dim3(BG_THREADS),
                     4 * BG_TILE_BYTES, st, A, W, nullptr, static_cast<uint16_t *>(out), nullptr, nullptr, 0, N, K,
                     epi, 0, tiles_n, 0, K / BG_BK, ga);
  return hipGetLastError();
}

hipError_t launch_gemm_grouped(const uint16_t *A, int a_nrows, const int32_t *a_rows, const uint16_t *W, void *out,
                               bool f32_out, const int32_t *tiles, const int32_t *n_tiles, int max_tiles, int N, int K,
                               int epi, hipStream_t st) {
  if (max_tiles <= 0) return hipSuccess;
  const int col_tiles = (logical_cols(N, epi) + SK_BN - 1) / SK_BN;
  const dim3 grid((unsigned)max_tiles * (unsigned)col_tiles);
  if (f32_out)
    hipLaunchKernelGGL(k_gemm_grouped<true>, grid, dim3(256), SK_LDS, st, A, a_nrows, a_rows, W, out, tiles, n_tiles,
                       max_tiles, N, K, epi, col_tiles);
  else
    hipLaunchKernelGGL(k_gemm_grouped<false>, grid, dim3(256), SK_LDS, st, A, a_nrows, a_rows, W, out, tiles,
                       n_tiles, max_tiles, N, K, epi, col_tiles);
  return hipGetLastError();
}

}  // namespace eb
