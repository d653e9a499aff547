// gfx950 (MI355X) kernels for ShallowStream's query-time evidence retrieval.
//
// Retrieval pipeline (Sec. 4.2 "Optional Evidence Retrieval"), all on one HIP
// stream, no host synchronisation:
//   k_prep      mean query per (layer, head), pre-scaled, split into bf16 hi+lo
//               and laid out as the MFMA B operand (lane-native).
//   k_sample    scores of an evenly spread sample of rows per list group
//               (k_score<SAMPLE> in head mode 1).  k_prep_sample does both
//               steps in one launch when its blocks fit one round.
//   k_thresh    per list, the r-th largest sample score: the streaming cut-off.
//               k_prep_thresh does prep, sample and cut-off in one launch for
//               short samples (one block per list).
//   k_stream    THE HOT KERNEL: streams every bf16 key row from HBM once.
//               The 16-row tiles of all lists form one sequence, cut into
//               XCD-weighted group ranges (plus a handed-out tail on
//               segment-rich batches); each tile comes in as coalesced
//               nontemporal 16-byte buffer loads, is swizzled through LDS into
//               the MFMA A layout, is scored by bf16 MFMA 16x16x32 against the
//               group's query columns (hi and lo parts, fp32 accumulation), and
//               rows at or above the cut-off are staged in LDS as 64-bit
//               composite keys and flushed with one atomic per (wave, column).
//               k_stream_hm is the same pass for head mode 1 (one list per
//               layer, the scores averaged over all query heads).
//   k_select    exact top-k per list from its candidates (radix selection over
//               the value range, items in registers, ties by row); a list whose
//               candidate count left [k, capacity] recomputes all of its scores
//               and selects exactly from them instead.  Each list then adds its
//               selected rows up per frame (count, fixed-point score sum).
//               k_select_dense runs two blocks per CU for many lists.
//   k_votes_pool  per stream, the vote-ranked pool from the frames' votes and
//               fixed-point attention mass: a vote histogram fixes the cut,
//               frames tied at it are ranked by counting (a radix cut over the
//               128-bit records when many tie), the pool is ranked by counting.
//   k_gram      fp32 Gram matrix of the pool descriptors.  k_pool_gram does
//               both in one launch (every Gram block ranks the pool itself)
//               when a stream's records fit in LDS.
//   k_maxmin    greedy max-min diversity over the Gram matrix.
//
// Append: k_unit_means (pooled keys and the Eq. memory_key descriptor), k_copy (raw rows) or k_kmeans
// (per-frame k-means compression).
//
// Ordering conventions: a score s maps to an order-preserving uint32 u(s); the
// composite key (u(s) << 32) | (0xFFFFFFFF - row) sorts descending exactly as
// (score desc, row asc), the top-k tie rule.
#include "ss_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdint>
#include <utility>

namespace ss {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kSelItems = 8;        // candidates per thread (of 1024) held in registers by k_select
constexpr int kThrItems = 16;       // sample scores per thread (of 1024) in k_thresh: 16384, the planner's bound
constexpr int kVoteLds = 4096;      // frames whose votes/mass live in LDS
constexpr int kPoolSort = 4096;     // records per pool sorting round
constexpr int kGramLdsPool = 128;   // pools up to this size keep their Gram matrix in LDS
constexpr int kMaxDescDim = 1024;
constexpr int kProbMassExp = 50;    // fixed-point exponent of attention-probability masses
constexpr int kBelowExp = 40;       // fixed-point exponent of the exp sums below a cut-off

// ---------------------------------------------------------------------------
// Small device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ord_u32(float s) {
  const uint32_t b = __float_as_uint(s);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float ord_f32(uint32_t u) {
  const uint32_t b = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(b);
}
__device__ __forceinline__ uint64_t mk_key(uint32_t u, uint32_t row) {
  return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - row);
}
__device__ __forceinline__ uint32_t key_row(uint64_t k) { return 0xFFFFFFFFu - (uint32_t)k; }
__device__ __forceinline__ float key_score(uint64_t k) { return ord_f32((uint32_t)(k >> 32)); }

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// The score arithmetic of every head-mode-0 path (sample, stream, exact
// recompute): one fp32 MFMA chain over the k-steps against the hi parts of the
// query mean, one against the lo parts, added at the end, so that each path
// gives a row the same bits.
template <int KS>
__device__ __forceinline__ f32x4 score_hilo(const u32x4 (&A)[KS], const u32x4 (&bh)[KS],
                                            const u32x4 (&bl)[KS]) {
  f32x4 h = {0.f, 0.f, 0.f, 0.f}, l = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < KS; ++i) h = mfma_bf16(A[i], bh[i], h);
#pragma unroll
  for (int i = 0; i < KS; ++i) l = mfma_bf16(A[i], bl[i], l);
  return h + l;
}

constexpr int kAuxNT = 2;  // buffer-load cache policy: nontemporal

__device__ __forceinline__ u32x4 ld_nt(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Head mode 1 (the layer's head-averaged score).  One B tile holds every KV
// head g of the layer: the hi part of its pre-scaled group query sum in column
// g and the lo part in column g + 8 (H_kv <= 8).  A tile of head g's keys is
// scored against it with one chain of MFMAs over the k-steps; lane (c, kg)
// keeps the result of head c mod 8, and a row's score is the sum over the 16
// columns in a fixed butterfly, read from column 0.  The sample, stream and
// exact-recompute paths all take these steps, so a row gets the same bits in
// each.
template <int KS>
__device__ __forceinline__ void hm_load_b(const u32x4* qb_layer, int Hk, u32x4 (&b)[KS]) {
  const int lane = threadIdx.x & 63, c = lane & 15, kg = lane >> 4, g = c & 7;
#pragma unroll
  for (int i = 0; i < KS; ++i)
    b[i] = g < Hk ? qb_layer[(size_t)g * (2 * KS * 64) + ((c < 8 ? 0 : KS) + i) * 64 + 16 * kg]
                  : u32x4{0, 0, 0, 0};
}

template <int KS>
__device__ __forceinline__ void hm_accumulate(const u32x4 (&A)[KS], const u32x4 (&b)[KS], int g, f32x4& v) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < KS; ++i) acc = mfma_bf16(A[i], b[i], acc);
  if (((threadIdx.x & 15) & 7) == g) v = acc;
}

#define SS_DPP_F(x, ctrl) __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), ctrl, 0xF, 0xF, false))
__device__ __forceinline__ f32x4 hm_finish(f32x4 v) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float x = v[j];
    x += SS_DPP_F(x, 0xB1);    // quad_perm 1,0,3,2
    x += SS_DPP_F(x, 0x4E);    // quad_perm 2,3,0,1
    x += SS_DPP_F(x, 0x124);   // row_ror 4
    x += SS_DPP_F(x, 0x128);   // row_ror 8
    v[j] = x;
  }
  return v;
}
#undef SS_DPP_F

// Exclusive prefix count of `p` among the lanes of a wave.
__device__ __forceinline__ int wave_excl_count(bool p) {
  const uint64_t m = __ballot(p);
  const int lane = threadIdx.x & (kWave - 1);
  return __popcll(m & ((1ull << lane) - 1ull));
}

// Inclusive prefix sum over the lanes of a wave (lane 0 first): DPP row_shr
// steps of 1, 2, 4 and 8 within each row of 16 lanes, then the totals of the
// rows below, read from lanes 15, 31 and 47.
__device__ __forceinline__ uint32_t wave_prefix_u32(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);   // row_shr 1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);   // row_shr 2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);   // row_shr 4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);   // row_shr 8
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)v, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)v, 47);
  const int row = (int)(threadIdx.x & (kWave - 1)) >> 4;
  return v + (row > 0 ? r0 : 0u) + (row > 1 ? r1 : 0u) + (row > 2 ? r2 : 0u);
}

// Inclusive suffix sum over the lanes of a wave (the lane and every higher one).
__device__ __forceinline__ uint32_t wave_suffix_u32(uint32_t v) {
  const uint32_t p = wave_prefix_u32(v);
  return (uint32_t)__builtin_amdgcn_readlane((int)p, kWave - 1) - p + v;
}

// Block-wide exclusive scan of `v`; `sh` needs blockDim/64 + 1 ints.  Returns the
// thread's exclusive prefix; `total` receives the block sum.
__device__ int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int x = (int)wave_prefix_u32((uint32_t)v);   // inclusive, wraps like int adds
  if (lane == kWave - 1) sh[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < nw; ++i) { const int t = sh[i]; sh[i] = run; run += t; }
    sh[nw] = run;
  }
  __syncthreads();
  const int r = sh[w] + x - v;
  total = sh[nw];
  __syncthreads();
  return r;
}

// Block argmax of (v, idx): larger v wins, then smaller idx.  `shv`/`shi` need
// blockDim/64 entries.  Every thread gets the winning index.
__device__ int block_argmax(float v, int idx, float* shv, int* shi) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(v, o);
    const int i2 = __shfl_xor(idx, o);
    if (v2 > v || (v2 == v && i2 < idx)) { v = v2; idx = i2; }
  }
  if (lane == 0) { shv[w] = v; shi[w] = idx; }
  __syncthreads();
  float bv = shv[0];
  int bi = shi[0];
  for (int i = 1; i < nw; ++i) {
    if (shv[i] > bv || (shv[i] == bv && shi[i] < bi)) { bv = shv[i]; bi = shi[i]; }
  }
  __syncthreads();
  return bi;
}

__device__ float block_max(float v, float* sh) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
  for (int i = 1; i < nw; ++i) r = fmaxf(r, sh[i]);
  __syncthreads();
  return r;
}

// Wave 0 finds, in a 256-bin histogram scanned from the top bin down, the bin
// holding the `need`-th element.  Writes bin, count above it and the bin count
// to res[0..2].
__device__ void find_digit(const uint32_t* hist, uint32_t need, uint32_t* res) {
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const uint32_t h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2],
                   h3 = hist[4 * lane + 3];
    const uint32_t mine = h0 + h1 + h2 + h3;
    const uint32_t x = wave_suffix_u32(mine);  // inclusive suffix sum over lanes >= lane
    const uint32_t above = x - mine;  // elements in bins of higher lanes
    if (above < need && need <= above + mine) {
      uint32_t a = above;
      const uint32_t hs[4] = {h0, h1, h2, h3};
      for (int j = 3; j >= 0; --j) {
        if (need <= a + hs[j]) {
          res[0] = 4 * lane + j;
          res[1] = a;
          res[2] = hs[j];
          break;
        }
        a += hs[j];
      }
    }
  }
  __syncthreads();
}

// Place of bin b in a histogram padded with one word after every 32 bins, so
// that the 64 lanes reading their own 32 consecutive bins start in 32
// different banks.
__device__ __forceinline__ uint32_t pad32(uint32_t b) { return b + (b >> 5); }

// Wave 0 finds, in an NB-bin histogram (NB = 64 * BPL) scanned from the top
// bin down, the bin holding the `need`-th element: res[0..2] = bin, count
// above it, bin count.  PAD: the histogram is laid out by pad32 (BPL = 32).
// Ends with a barrier.
template <int BPL, bool PAD = false>
__device__ void find_digit_wide(const uint32_t* hist, uint32_t need, uint32_t* res) {
  static_assert(!PAD || BPL == 32, "padded histograms hold 32 bins per lane");
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const uint32_t* hl = hist + (PAD ? (BPL + 1) : BPL) * lane;
    uint32_t hs[BPL], mine = 0;
#pragma unroll
    for (int j = 0; j < BPL; ++j) { hs[j] = hl[j]; mine += hs[j]; }
    const uint32_t x = wave_suffix_u32(mine);  // inclusive suffix sum over lanes >= lane
    const uint32_t above = x - mine;
    if (above < need && need <= above + mine) {
      uint32_t a = above;
      for (int j = BPL - 1; j >= 0; --j) {
        if (need <= a + hs[j]) {
          res[0] = BPL * lane + j;
          res[1] = a;
          res[2] = hs[j];
          break;
        }
        a += hs[j];
      }
    }
  }
  __syncthreads();
}

// r-th largest (1-based) of n uint32 values given by get(i).  Returns it and the
// number of values strictly greater.  hist: LDS [256]; res: LDS [4].
template <class Get>
__device__ uint32_t radix_select_u32(Get get, int n, uint32_t r, uint32_t* hist, uint32_t* res,
                                     uint32_t& n_greater) {
  uint32_t prefix = 0, mask = 0, need = r;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint32_t v = get(i);
      if ((v & mask) == prefix) atomicAdd(&hist[(v >> shift) & 255u], 1u);
    }
    __syncthreads();
    find_digit(hist, need, res);
    prefix |= res[0] << shift;
    mask |= 255u << shift;
    need -= res[1];
    __syncthreads();
  }
  n_greater = r - need;
  return prefix;
}

// r-th largest of n distinct uint64 keys; stops as soon as a whole bucket is
// selected.  Returns a threshold t such that exactly r keys are >= t.
template <class Get>
__device__ uint64_t radix_select_u64(Get get, int n, uint32_t r, uint32_t* hist, uint32_t* res) {
  uint64_t prefix = 0, mask = 0;
  uint32_t need = r;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint64_t v = get(i);
      if ((v & mask) == prefix) atomicAdd(&hist[(uint32_t)(v >> shift) & 255u], 1u);
    }
    __syncthreads();
    find_digit(hist, need, res);
    const uint32_t b = res[0], above = res[1], inb = res[2];
    __syncthreads();
    prefix |= (uint64_t)b << shift;
    mask |= 255ull << shift;
    need -= above;
    if (inb == need) break;  // the whole bucket is taken: prefix (low bits 0) is the cut
  }
  return prefix;
}

// Threshold (hi, lo) such that exactly r of the n distinct 128-bit keys
// get(i) = (hi, lo) compare >= it; same early exit as radix_select_u64.
template <class Get>
__device__ void radix_select_u128(Get get, int n, uint32_t r, uint32_t* hist, uint32_t* res,
                                  uint64_t& cut_hi, uint64_t& cut_lo) {
  uint64_t ph = 0, pl = 0, mh = 0, ml = 0;
  uint32_t need = r;
  for (int d = 0; d < 16; ++d) {
    const int shift = 56 - 8 * (d & 7);
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      uint64_t h, l;
      get(i, h, l);
      if ((h & mh) == ph && (l & ml) == pl)
        atomicAdd(&hist[(uint32_t)((d < 8 ? h : l) >> shift) & 255u], 1u);
    }
    __syncthreads();
    find_digit(hist, need, res);
    const uint32_t b = res[0], above = res[1], inb = res[2];
    __syncthreads();
    if (d < 8) { ph |= (uint64_t)b << shift; mh |= 255ull << shift; }
    else { pl |= (uint64_t)b << shift; ml |= 255ull << shift; }
    need -= above;
    if (inb == need) break;
  }
  cut_hi = ph;
  cut_lo = pl;
}

// Descending bitonic sort of n (power of two) uint64 keys in LDS.
__device__ void bitonic_desc_u64(uint64_t* a, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < (n >> 1); i += blockDim.x) {
        const int lo = 2 * j * (i / j) + (i % j), hi = lo + j;
        const bool desc = (lo & k) == 0;
        const uint64_t x = a[lo], y = a[hi];
        if (desc ? (x < y) : (x > y)) { a[lo] = y; a[hi] = x; }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ bool rec_less(uint64_t ah, uint64_t al, uint64_t bh, uint64_t bl) {
  return ah < bh || (ah == bh && al < bl);
}

// Descending bitonic sort of n (power of two) 128-bit records (hi, lo) in LDS.
__device__ void bitonic_desc_u128(uint64_t* hi, uint64_t* lo, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < (n >> 1); i += blockDim.x) {
        const int a = 2 * j * (i / j) + (i % j), b = a + j;
        const bool desc = (a & k) == 0;
        const uint64_t xh = hi[a], xl = lo[a], yh = hi[b], yl = lo[b];
        const bool sw = desc ? rec_less(xh, xl, yh, yl) : rec_less(yh, yl, xh, xl);
        if (sw) { hi[a] = yh; lo[a] = yl; hi[b] = xh; lo[b] = xl; }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int pow2_ceil(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// ---------------------------------------------------------------------------
// k_prep: query mean -> MFMA B operand (bf16 hi + lo)
// ---------------------------------------------------------------------------
struct PrepArgs {
  int Hq, Hk, G, L, head_mode;
  int first;       // first (stream, layer) pair of this launch: pair = s * L + l
  const uint16_t* q[128];
  int nq[kMaxStreams];
  float qscale[kMaxStreams];
  u32x4* qB;       // [S][L][H_kv][2][D/32][64]
  float* qcol;     // [S][L][H_kv][16] L1 norm of each scaled B column, or null
};

// Query token groups of the B-tile prep (the partial sums of each are added in
// group order).
constexpr int kPrepGroups = 4;

// Forms the B tile of (pair, KV head g) with the block's 8 D threads; `part`
// is the block's LDS scratch for the token-group partial sums.  The threads of
// token group 0 (the first 2 D threads, whole waves) hold the result: they
// write it to `out_lds` if given, and to the global B tile and the column L1
// norms if `global` is set.
template <int D>
__device__ __forceinline__ void prep_b(const PrepArgs& a, int pair_local, int g,
                                       float (*part)[2 * D][8], u32x4* out_lds, bool global) {
  constexpr int KS = D / 32, NE = D / 8, NT = 2 * D;  // NT threads per token group
  const int pair = a.first + pair_local;
  const int s = pair / a.L;
  const uint16_t* q = a.q[pair_local];
  const int nq = a.nq[s];
  const float scale = a.qscale[s];
  const int tg = threadIdx.x / NT, t = threadIdx.x % NT;
  const int col = t / NE, ec = t % NE;
  int h0, h1;
  if (a.head_mode == 0) {
    h0 = g * a.G + col;
    h1 = (col < a.G) ? h0 + 1 : h0;
  } else {
    h0 = g * a.G;
    h1 = (col == 0) ? h0 + a.G : h0;
  }
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int e0 = 8 * ec;
  for (int h = h0; h < h1; ++h) {
    const uint16_t* qh = q + (size_t)h * nq * D + e0;
    // tokens tg, tg + 4, ... in increasing order; 16 loads in flight per pass,
    // from clamped in-bounds token indices (only tokens below nq are added)
    for (int j0 = tg; j0 < nq; j0 += 16 * kPrepGroups) {
      u32x4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        v[u] = *reinterpret_cast<const u32x4*>(qh + (size_t)min(j0 + u * kPrepGroups, nq - 1) * D);
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (j0 + u * kPrepGroups < nq) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            acc[2 * w] += bf16_lo(v[u][w]);
            acc[2 * w + 1] += bf16_hi(v[u][w]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int w = 0; w < 8; ++w) part[tg][t][w] = acc[w];
  __syncthreads();
  if (tg == 0) {
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      float x = part[0][t][w];
      for (int k = 1; k < kPrepGroups; ++k) x += part[k][t][w];
      acc[w] = x;
    }
    u32x4 hi, lo;
    float l1 = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float x0 = acc[2 * w] * scale, x1 = acc[2 * w + 1] * scale;
      l1 += fabsf(x0) + fabsf(x1);
      const uint16_t a0 = bf16_rne(x0), a1 = bf16_rne(x1);
      const uint16_t b0 = bf16_rne(x0 - __uint_as_float((uint32_t)a0 << 16));
      const uint16_t b1 = bf16_rne(x1 - __uint_as_float((uint32_t)a1 << 16));
      hi[w] = (uint32_t)a0 | ((uint32_t)a1 << 16);
      lo[w] = (uint32_t)b0 | ((uint32_t)b1 << 16);
    }
    const int i = ec >> 2, lane = col + 16 * (ec & 3);
    if (out_lds) {
      out_lds[(0 * KS + i) * kWave + lane] = hi;
      out_lds[(1 * KS + i) * kWave + lane] = lo;
    }
    if (global) {
      u32x4* out = a.qB + ((size_t)pair * a.Hk + g) * (2 * KS * kWave);
      out[(0 * KS + i) * kWave + lane] = hi;
      out[(1 * KS + i) * kWave + lane] = lo;
    }
    // the NE threads of a column are adjacent lanes of one wave
#pragma unroll
    for (int o = NE / 2; o > 0; o >>= 1) l1 += __shfl_xor(l1, o);
    if (global && a.qcol && ec == 0) a.qcol[((size_t)pair * a.Hk + g) * 16 + col] = l1;
  }
}

// One block of 8*D threads per (stream, layer, KV head): thread (tg, col, ec)
// sums, over the query tokens j = tg mod 4, dims 8 ec .. 8 ec + 7 of B-tile
// column col; the four partial sums are then added in tg order.  In the
// lane-native layout those dims belong to k-step i = ec / 4 of lane
// col + 16 (ec % 4).  Column c of head-mode 0 is query head g*G + c; head-mode 1
// uses column 0 only, holding the sum of the group's head means (the layer's
// head average is the sum over KV heads of these columns against their keys).
template <int D>
__global__ __launch_bounds__(8 * D) void k_prep(PrepArgs a) {
  __shared__ float part[kPrepGroups][2 * D][8];
  prep_b<D>(a, blockIdx.x / a.Hk, blockIdx.x % a.Hk, part, nullptr, true);
}

// ---------------------------------------------------------------------------
// k_score: the MFMA scoring core in three roles
// ---------------------------------------------------------------------------
enum { K_SAMPLE = 0, K_STREAM = 1, K_FULL = 2 };

struct ScoreArgs {
  int L, Hq, Hk, G, NL, ngs, head_mode;
  int chunk;                          // units (rows or sample slots) per item
  int total_items;
  int S;
  const uint16_t* keys[kMaxStreams];  // arena keys of each stream
  int32_t stride[kMaxStreams];        // rows per (layer, KV head) in the arena
  int32_t n[kMaxStreams];             // candidate rows
  int32_t units[kMaxStreams];         // enumerated units per (layer, set)
  int32_t item_base[kMaxStreams + 1];
  const u32x4* qB;
  // K_SAMPLE
  float* samp;
  int samp_stride;
  int64_t samp_step[kMaxStreams];     // n 2^32 / m: sample u sits at row (u step + step/2) >> 32
  // K_STREAM
  int score_mode;                      // 1: attention probabilities (exp sums below each cut-off)
  uint64_t* below;                     // fixed-point sums of exp below each cut-off
  const float* lhat;                   // hm_prob: log-sum-exp estimate of each (stream, layer, head)
  uint32_t* left_max;                  // hm_prob: largest alpha_hat per list among the rows left out
  const uint32_t* tau;
  uint32_t* cnt;
  uint64_t* cand;
  int cap;
  int64_t tile_base[kMaxStreams + 1];  // first tile of each stream; tiles of all streams in a row
  int32_t ntile[kMaxStreams];          // 16-row tiles per (layer, KV head) segment
  int sgroup;                          // blocks per XCD group of the streaming pass
  int xcd_weights;                     // weight the group ranges by XCD parity (MI355X with all 256 CUs)
  int64_t dyn_tiles;                   // the last tiles, handed out in chunks (0: all static)
  int dyn_chunk;                       // tiles per handed-out chunk
  uint32_t* dyn_ctr;                   // kDynCtr chunk counters, kDynStride words apart
  // K_FULL (parity scores of one list)
  int only_list;
  float* full;
  int64_t full_base[kMaxStreams];
  int32_t full_stride[kMaxStreams];
  int64_t row0;
};

// Evenly spread sample: sample u of m sits at row ((u + 1/2) n / m) rounded
// down, in 32.32 fixed point; the identity when m == n.
__device__ __forceinline__ int64_t sample_row(int64_t step, int u) {
  return (int64_t)(((uint64_t)u * (uint64_t)step + ((uint64_t)step >> 1)) >> 32);
}

// Row of the key index scored for unit u of stream s.
template <int KIND>
__device__ __forceinline__ int64_t unit_row(const ScoreArgs& a, int s, int u) {
  if (KIND == K_SAMPLE) return sample_row(a.samp_step[s], u); else if (KIND == K_FULL) {
    return a.row0 + u;
  } else {
    return u;
  }
}

// Per-lane output of one 16-row tile: lane (col, kg) holds the scores of rows
// 4 kg + j (j < 4) of the tile for output column col.  Called by whole waves.
// K_SAMPLE writes sample scores, K_FULL whole score rows.
template <int KIND>
__device__ __forceinline__ void emit(const ScoreArgs& a, int s, int list, bool colv, bool wr,
                                     int tile_u0, int u1, f32x4 acc, int kg) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int u = tile_u0 + 4 * kg + j;
    const float sc = acc[j] + 0.0f;
    if (KIND == K_SAMPLE) {
      if (colv && u < u1) a.samp[(size_t)list * a.samp_stride + u] = sc;
    } else {
      if (wr && u < u1) {
        const int ll = list - s * a.NL;
        a.full[a.full_base[s] + (int64_t)ll * a.full_stride[s] + u] = sc;
      }
    }
  }
}

// The value of lane ^ 16 / lane ^ 32 (whole wave active): gfx950's row swaps
// exchange rows of 16 lanes in registers.
__device__ __forceinline__ int lane_xor16(int x) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return ((threadIdx.x >> 4) & 1) ? (int)r[0] : (int)r[1];
}
__device__ __forceinline__ int lane_xor32(int x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return ((threadIdx.x >> 5) & 1) ? (int)r[0] : (int)r[1];
}

// Candidates of the streaming pass wait in LDS, kStage per (wave, column), and
// go to the list's global buffer in one flush: one global atomic per (wave,
// column, flush) keeps returning atomics out of the tile loop (a full stage
// flushes here; at a segment end k_stream flushes a whole block at once,
// block_flush below).  `lc` is the
// staged count of the lane's column, the same in the column's four lanes.
// The waves whose range crosses a frame where most rows pass (the frames that
// collect the votes) flush most and finish last; 64 keys per column instead of
// 32 took the 1-hour pass from 413 to 405 us (32 KiB of stage per block, two
// blocks per CU).
constexpr int kStage = 64;

// Query heads a probability streaming pass can hold (H_kv * d <= 512 and
// G <= 16: H_q <= 128).
constexpr int kHpHeads = 128;

__device__ __forceinline__ void stage_flush(const ScoreArgs& a, int list, bool colv, int col, int kg,
                                            const uint64_t* st, int& lc) {
  __builtin_amdgcn_wave_barrier();
  int base = 0;   // set in the column's kg = 0 lane only, then summed over its four lanes
  if (kg == 0 && colv && lc > 0) base = (int)atomicAdd(&a.cnt[list], (uint32_t)lc);
  base += lane_xor16(base);
  base += lane_xor32(base);
  for (int e = kg; e < lc; e += 4) {
    const uint32_t slot = (uint32_t)base + (uint32_t)e;
    if (slot < (uint32_t)a.cap) a.cand[(size_t)list * a.cap + slot] = st[col * kStage + e];
  }
  __builtin_amdgcn_wave_barrier();
  lc = 0;
}

// Rows of a tile at or above the cut-off are staged as composite keys.  Lane
// (col, kg) holds rows 4 kg + j of the tile for column col.  Compared as
// floats: for finite scores x >= ord_f32(tau) selects exactly the rows whose
// canonical key ord_u32(x + 0) is at least tau (-0 and +0 compare equal and
// share one key); invalid columns carry a NaN cut-off, which nothing passes.
__device__ __forceinline__ void stream_emit(const ScoreArgs& a, int list, bool colv, int col,
                                            float tau_f, int tile_u0, int u1, f32x4 acc, int kg,
                                            uint64_t* st, int& lc, double& below, bool prob) {
  bool pass[4];
  int c = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool valid = tile_u0 + 4 * kg + j < u1;
    pass[j] = valid && acc[j] >= tau_f;
    c += pass[j];
    // attention probabilities: every row below the cut-off adds exp(s - tau),
    // in (0, 1), to its list's normaliser
    if (prob && colv && valid && !pass[j]) below += (double)__expf(acc[j] - tau_f);
  }
  if (__ballot(c > 0) == 0) return;
  // the column's four lanes (lanes col + 16 kg) agree on a slot range, in kg
  // order; their counts travel by row swaps in registers
  const int c16 = lane_xor16(c);
  const int c32 = lane_xor32(c);
  const int c48 = lane_xor32(c16);
  const int total = c + c16 + c32 + c48;
  const int prefix = kg == 0 ? 0 : kg == 1 ? c16 : kg == 2 ? c32 + c48 : c16 + c32 + c48;
  if (__any(lc + total > kStage)) stage_flush(a, list, colv, col, kg, st, lc);
  int slot = lc + prefix;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (pass[j]) {
      st[col * kStage + slot] = mk_key(ord_u32(acc[j] + 0.0f), (uint32_t)(tile_u0 + 4 * kg + j));
      ++slot;
    }
  }
  lc += total;
}

// Adds a (wave, column)'s sum of exp below the cut-off to the list's fixed-point
// total at the end of a segment visit: the column's four lanes are added in a
// fixed order, scaled by 2^kBelowExp and rounded, and integer atomics keep the
// total independent of the order of the visits.  Called by the whole wave.
__device__ __forceinline__ void below_flush(uint64_t* dst, bool colv, int kg, double& v, double scale) {
  double x = v;
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  if (kg == 0 && colv && x > 0.0)
    atomicAdd(reinterpret_cast<unsigned long long*>(dst), (unsigned long long)llrint(ldexp(x * scale, kBelowExp)));
  v = 0.0;
}

// The end of a segment visit for a whole block of k_stream: every wave calls
// it at the same segment end (the waves of a group walk the same segments).
// The waves of a group end a segment together, and their atomics on a list's
// counter queue one behind the other at the memory side (returning or not:
// with one per wave, C3's pass took 6 us and C4's 5 us longer than with none).
// One per (block, column) shortens that queue fourfold: per call, C3 56.4 ->
// 51.6 us, C2 110.9 -> 109.2 us, C4 449.8 -> 446.2 us, C5 2,000 -> 1,995 us
// (the head-mean pass, with one list per layer and few keys per wave, did not
// gain; the probability pass groups its per-head sums the same way).  Each
// wave's keys go to the block's slot range after those of the lower waves.
// With `prob`, each wave's exp sum below the cut-off is rounded to fixed point
// as in below_flush and the block adds the integers, so the total does not
// depend on how the sums are grouped.
template <int NW>
struct FlushShared {
  uint32_t cnt[NW][16];          // staged keys per (wave, column)
  uint32_t base[16];             // the column's first slot
  unsigned long long below[16];  // the column's fixed-point exp sum (zero between flushes)
};

template <int NW>
__device__ __forceinline__ void block_flush(const ScoreArgs& a, int list, bool colv, int col, int kg, int wave,
                                            const uint64_t* st, int& lc, bool prob, double& bsum,
                                            FlushShared<NW>& fl) {
  if (kg == 0) fl.cnt[wave][col] = colv ? (uint32_t)lc : 0u;
  if (prob) {
    double x = bsum;
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if (kg == 0 && colv && x > 0.0) atomicAdd(&fl.below[col], (unsigned long long)llrint(ldexp(x, kBelowExp)));
    bsum = 0.0;
  }
  __syncthreads();
  if (wave == 0 && kg == 0 && colv) {
    uint32_t tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) tot += fl.cnt[w][col];
    fl.base[col] = tot ? atomicAdd(&a.cnt[list], tot) : 0u;
    if (prob) {
      const unsigned long long b = fl.below[col];
      if (b) atomicAdd(reinterpret_cast<unsigned long long*>(&a.below[list]), b);
      fl.below[col] = 0;
    }
  }
  __syncthreads();
  uint32_t base = fl.base[col];
  for (int w = 0; w < wave; ++w) base += fl.cnt[w][col];
  for (int e = kg; e < lc; e += 4) {
    const uint32_t slot = base + (uint32_t)e;
    if (slot < (uint32_t)a.cap) a.cand[(size_t)list * a.cap + slot] = st[col * kStage + e];
  }
  lc = 0;
  __syncthreads();   // the tables are rewritten at the next segment end
}

// Head-mode 0: one KV head per item, its G query heads in the MFMA columns, the
// B operand in registers, PF tiles in flight per wave.
template <int D, int KIND>
__global__ __launch_bounds__(256) void k_score(ScoreArgs a) {
  static_assert(KIND != K_STREAM, "head-mode-0 streaming runs in k_stream");
  constexpr int KS = D / 32, PF = 2;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  for (int item = blockIdx.x; item < a.total_items; item += gridDim.x) {
    int s = 0;
    while (item >= a.item_base[s + 1]) ++s;
    const int rem = item - a.item_base[s];
    const int units = a.units[s];
    const int nch = (units + a.chunk - 1) / a.chunk;
    const int chunk = rem % nch, lg = rem / nch;
    const int g = lg % a.ngs, l = lg / a.ngs;
    const int u0 = chunk * a.chunk, u1 = min(units, u0 + a.chunk);
    const bool colv = col < a.G;
    const int list = s * a.NL + l * a.Hq + g * a.G + col;
    bool wr = false;
    if (KIND == K_FULL) {
      const int ll = l * a.Hq + g * a.G + col;
      wr = colv && ll == a.only_list;
      if (!__any(wr)) continue;  // same decision in every wave of the block
    }
    const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * a.Hk + g) * (2 * KS * kWave);
    u32x4 bh[KS], bl[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      bh[i] = qb[i * kWave + lane];
      bl[i] = qb[(KS + i) * kWave + lane];
    }
    const uint16_t* base = a.keys[s] + ((size_t)l * a.Hk + g) * (size_t)a.stride[s] * D + 8 * kg;
    const int ntiles = (u1 - u0 + kTile - 1) / kTile;

    auto load = [&](int t, u32x4 (&A)[KS]) {
      const int u = u0 + t * kTile + rl;
      const bool ok = (t < ntiles) && (u < u1);
      const int64_t row = ok ? unit_row<KIND>(a, s, u) : 0;
      const uint16_t* p = base + row * D;
#pragma unroll
      for (int i = 0; i < KS; ++i) A[i] = ok ? ld_nt(p + 32 * i) : u32x4{0, 0, 0, 0};
    };

    u32x4 A[PF][KS];
#pragma unroll
    for (int p = 0; p < PF; ++p) load(wave + p * nw, A[p]);
    for (int t = wave; t < ntiles; t += PF * nw) {
#pragma unroll
      for (int p = 0; p < PF; ++p) {
        const int tt = t + p * nw;
        if (tt < ntiles) {
          const f32x4 acc = score_hilo<KS>(A[p], bh, bl);
          emit<KIND>(a, s, list, colv, wr, u0 + tt * kTile, u1, acc, kg);
        }
        load(tt + PF * nw, A[p]);
      }
    }
  }
}

// Tiles of the streaming passes are numbered one after another over all
// segments.  `sgroup` blocks of one XCD (blocks are dealt to the 8 XCDs in
// turn) share one contiguous range of that numbering, and their 4 sgroup waves
// take its tiles in turn, so that at any moment the group reads one window of
// about 4 sgroup tiles.  Measured on the 1-hour workload, a few dozen such
// windows in flight read HBM faster than one private range per wave
// (thousands of scattered streams) or one sweep by the whole grid: 32 blocks
// per group (16 windows) beat 8 (64 windows) by 2%.  But every wave visits
// every segment of its group's range, and at the end of each visit it flushes
// its staged candidates with a returning atomic on the list's counter that all
// the group's waves hit at about the same moment.  Where segments are short
// against the range (the 16-stream ragged batch: 192 segments, 12 per range at
// 32 blocks) those stalls cost 10% of the pass, and 8 blocks per group (3
// segments per range) took it from 2,060 to 1,964 us.  The host therefore
// takes the largest group of at most kStreamGroupMax blocks whose range spans
// at most three average segments.
constexpr int kStreamGroupMax = 32;

// Share of the tiles per group by XCD parity.  On this part the odd XCDs read
// HBM about 9% slower than the even ones while all eight stream (the same
// pattern on every box measured: with equal shares the even XCDs finish the
// 1-hour pass at 350-380 us and the odd ones at 386-417 us), so a group on an
// even XCD takes kXcdEvenWeight / kXcdOddWeight times the tiles of one on an odd
// XCD (on a device of 256 CUs, the whole MI355X, where block b runs on XCD
// b mod 8).  Measured: 1-hour pass 409 -> 403 us, 16-stream batch 1,954 -> 1,932 us;
// the XCD end times then no longer split by parity but still spread by about
// 20 us.  Handing the last 10-20% of the tiles out in chunks through atomic
// counters (below) cost the 1-hour pass 7-35 us, since single-wave chunks lose
// the DRAM locality of the group windows, so it is kept for the segment-rich
// batches only.  Only the split of the tiles between waves depends on these
// weights.
constexpr int64_t kXcdEvenWeight = 1090;
constexpr int64_t kXcdOddWeight = 1000;

// The handed-out tail of the streaming pass on batches of many short segments
// (where the group size rule picks fewer than kStreamGroupMax blocks): kDynCtr
// chunk counters, each in its own 256-byte line; kDynPermille of the tiles in
// chunks of kDynChunk.  On the 16-stream batch it took the pass from 1,950 to
// 1,895 us (the waves that visit many segments no longer finish last).
constexpr int kDynCtr = 32;
constexpr int kDynStride = 64;
constexpr int kDynPermille = 150;
constexpr int kDynChunk = 16;

struct WaveRange {
  int64_t b0, b1;   // the group's tiles
  int sw, wg;       // waves in the group, this wave's rank among them
};

__device__ __forceinline__ WaveRange wave_range(int64_t total, int wave, int sgroup, bool xcd_weights) {
  const int64_t nb = gridDim.x, b = blockIdx.x;
  int64_t ng, grp;
  int members, rank;
  if (nb % (8 * sgroup) == 0) {
    ng = nb / sgroup;
    const int64_t x = b % 8, r = b / 8;   // XCD, and rank among its blocks
    grp = (r / sgroup) * 8 + x;
    members = sgroup;
    rank = (int)(r % sgroup);
    // groups alternate even and odd XCDs; ng is a multiple of 8
    const int64_t even = xcd_weights ? kXcdEvenWeight : kXcdOddWeight;
    const int64_t pair = even + kXcdOddWeight;
    const int64_t w0 = (grp / 2) * pair + (grp % 2) * even;
    const int64_t w1 = w0 + ((grp % 2) ? kXcdOddWeight : even);
    const int64_t wt = (ng / 2) * pair;
    WaveRange w;
    w.b0 = total * w0 / wt;
    w.b1 = total * w1 / wt;
    w.sw = 4 * members;
    w.wg = rank * 4 + wave;
    return w;
  } else {
    ng = (nb + sgroup - 1) / sgroup;
    grp = b / sgroup;
    members = (int)min<int64_t>(sgroup, nb - grp * sgroup);
    rank = (int)(b - grp * sgroup);
  }
  WaveRange w;
  w.b0 = grp * total / ng;
  w.b1 = (grp + 1) * total / ng;
  w.sw = 4 * members;
  w.wg = rank * 4 + wave;
  return w;
}

// First tile of this wave at or after segment-local tile `tb`, the piece of
// the group's range that starts at flat tile T.
__device__ __forceinline__ int first_tile(const WaveRange& w, int64_t T, int tb) {
  const int d = (int)((T - w.b0) % w.sw);
  return tb + (w.wg - d + w.sw) % w.sw;
}

// Streaming pass, head-mode 0, over the group ranges above; the segment of a
// tile is a (stream, layer, KV head) list group.  A tile is read with coalesced 16-byte
// loads (one instruction covers 1 KiB of consecutive rows), stored into the
// wave's LDS tile and read back in the MFMA A layout.  LDS holds the tile as
// 256-byte lines of 16 chunks with chunk C of line R at position C ^ (R mod 16),
// which keeps both the row-major writes and the column reads free of bank
// conflicts.
template <int D>
__global__ __launch_bounds__(256) void k_stream(ScoreArgs a) {
  constexpr int CPR = D / 8;        // 16-byte chunks per key row
  constexpr int TCH = 16 * CPR;     // chunks per tile
  constexpr int NI = TCH / kWave;   // load instructions per tile
  constexpr int KS = D / 32;        // MFMA k-steps
  constexpr int PF = 128 / D;       // tiles in flight per wave
  __shared__ u32x4 tiles[4][TCH];
  __shared__ uint64_t stage[4 * kMaxGroup * kStage];
  __shared__ FlushShared<4> fl;
  if (threadIdx.x < 16) fl.below[threadIdx.x] = 0;
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: segment state in SGPRs
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  u32x4* lt_ = tiles[wave];
  uint64_t* st = stage + wave * kMaxGroup * kStage;
  // Tiles [0, total - dyn_tiles) in the wave's static share of its group's
  // range (see wave_range); then, on batches of many short segments, chunks of
  // the last dyn_tiles handed out by the chunk counters to whichever waves are
  // free (the waves that visit many segments flush more and fall behind).
  const int64_t total = a.tile_base[a.S], static_end = total - a.dyn_tiles;
  // bsync: every wave of the block walks the same segments (a group range),
  // so each segment visit ends in one flush for the whole block
  auto run_range = [&](const WaveRange& wr, bool bsync) {
    const int SW = wr.sw;
    for (int64_t T = wr.b0; T < wr.b1;) {
      int s = 0;
      while (T >= a.tile_base[s + 1]) ++s;
      const int64_t rem = T - a.tile_base[s];
      const int nt = a.ntile[s];
      const int lg = (int)(rem / nt);
      const int tb = (int)(rem - (int64_t)lg * nt);
      const int t1 = (int)min<int64_t>(nt, tb + (wr.b1 - T));
      const int t0 = first_tile(wr, T, tb);
      T += t1 - tb;
      if (t0 >= t1 && !bsync) continue;   // (in a block flush the wave takes part with no keys)
      const int g = lg % a.Hk, l = lg / a.Hk;
      const int n = a.n[s];
      const bool colv = col < a.G;
      const int list = s * a.NL + l * a.Hq + g * a.G + col;
      const float tau_f = ord_f32(colv ? a.tau[list] : 0xFFFFFFFFu);
      const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * a.Hk + g) * (2 * KS * kWave);
      u32x4 bh[KS], bl[KS];
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        bh[i] = qb[i * kWave + lane];
        bl[i] = qb[(KS + i) * kWave + lane];
      }
      // The segment is read through a buffer resource of exactly n rows: lanes
      // past the last row, and the loads that run ahead of the range, fetch
      // zeros without touching memory (the host keeps a segment below 2 GiB).
      // Lane q of load i covers the 16-byte chunk 64 i + q of the tile.
      const uint16_t* seg = a.keys[s] + ((size_t)l * a.Hk + g) * (size_t)a.stride[s] * D;
      const __amdgpu_buffer_rsrc_t rsrc =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(seg), (short)0, n * D * 2, 0x00020000);
      auto load = [&](int t, u32x4 (&V)[NI]) {
        const uint32_t off = t < t1 ? (uint32_t)t * (TCH * 16) + lane * 16 : 0x80000000u;
#pragma unroll
        for (int i = 0; i < NI; ++i)
          V[i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off + i * kWave * 16, 0, kAuxNT);
      };
      // The next loads are issued as soon as a tile's registers have gone to
      // LDS, so they overlap the MFMAs and the candidate test.  Every pass of
      // the loop body loads and computes (a pass past the range works on zeros
      // and emits nothing), which keeps the waits exact.
      u32x4 V[PF][NI];
#pragma unroll
      for (int p = 0; p < PF; ++p) load(t0 + SW * p, V[p]);
      int lc = 0;
      double bsum = 0.0;
      const bool prob = a.score_mode != 0;
      for (int t = t0; t < t1; t += SW * PF) {
#pragma unroll
        for (int p = 0; p < PF; ++p) {
          const int tt = t + SW * p;
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            const int q = i * kWave + lane, R = q >> 4, C = q & 15;
            lt_[R * 16 + (C ^ (R & 15))] = V[p][i];
          }
          __builtin_amdgcn_wave_barrier();
          load(tt + SW * PF, V[p]);
          u32x4 A[KS];
#pragma unroll
          for (int i = 0; i < KS; ++i) {
            const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
            A[i] = lt_[R * 16 + (C ^ (R & 15))];
          }
          __builtin_amdgcn_wave_barrier();
          const f32x4 acc = score_hilo<KS>(A, bh, bl);
          if (tt < t1) stream_emit(a, list, colv, col, tau_f, tt * kTile, n, acc, kg, st, lc, bsum, prob);
        }
      }
      if (bsync) {
        block_flush<4>(a, list, colv, col, kg, wave, st, lc, prob, bsum, fl);
      } else {
        if (__any(lc > 0)) stage_flush(a, list, colv, col, kg, st, lc);
        if (prob) below_flush(&a.below[list], colv, kg, bsum, 1.0);
      }
    }
  };
  run_range(wave_range(static_end, wave, a.sgroup, a.xcd_weights != 0), true);
  if (a.dyn_tiles > 0) {
    // K = min(kDynCtr, grid / 8) counters (at least one); counter k serves the
    // chunks k, k + K, ..., and block b uses counter (b / 8) mod K, so every
    // counter has blocks and the blocks that share one span all XCDs (block b
    // sits on XCD b mod 8)
    const int K = (int)min<int64_t>(kDynCtr, max<int64_t>(1, (int64_t)gridDim.x / 8));
    const int k0 = (int)((blockIdx.x >> 3) % K);
    uint32_t* ctr = a.dyn_ctr + k0 * kDynStride;
    const int64_t nch = (a.dyn_tiles + a.dyn_chunk - 1) / a.dyn_chunk;
    for (;;) {
      uint32_t q = 0;
      if (lane == 0) q = atomicAdd(ctr, 1u);
      q = __builtin_amdgcn_readfirstlane(q);
      const int64_t c = k0 + (int64_t)K * q;
      if (c >= nch) break;
      WaveRange d;
      d.b0 = static_end + c * a.dyn_chunk;
      d.b1 = min<int64_t>(d.b0 + a.dyn_chunk, total);
      d.sw = 1;
      d.wg = 0;
      run_range(d, false);
    }
  }
}

// Sample pass, head-mode 0: the m sampled rows of every (stream, layer, KV
// head) list group, 16 to a tile, numbered one after another and cut into one
// contiguous range per wave; a tile's rows are gathered with
// coalesced loads (16 lanes per 256-byte row, four rows per instruction) into
// the wave's LDS tile and scored with the same arithmetic as k_stream.
template <int D>
__global__ __launch_bounds__(256) void k_sample(ScoreArgs a) {
  constexpr int CPR = D / 8, TCH = 16 * CPR, NI = TCH / kWave, KS = D / 32;
  __shared__ u32x4 tiles[4][TCH];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  u32x4* lt_ = tiles[wave];
  const int64_t nw = (int64_t)gridDim.x * 4, gw = (int64_t)blockIdx.x * 4 + wave;
  const int64_t total = a.tile_base[a.S];
  const int64_t T1 = (gw + 1) * total / nw;
  int64_t T = gw * total / nw;
  while (T < T1) {
    int s = 0;
    while (T >= a.tile_base[s + 1]) ++s;
    const int64_t rem = T - a.tile_base[s];
    const int nt = a.ntile[s];
    const int lg = (int)(rem / nt);
    const int t0 = (int)(rem - (int64_t)lg * nt);
    const int t1 = (int)min<int64_t>(nt, t0 + (T1 - T));
    const int g = lg % a.Hk, l = lg / a.Hk;
    const int n = a.n[s], m = a.units[s];
    const int64_t step = a.samp_step[s];
    const bool colv = col < a.G;
    const int list = s * a.NL + l * a.Hq + g * a.G + col;
    const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * a.Hk + g) * (2 * KS * kWave);
    u32x4 bh[KS], bl[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      bh[i] = qb[i * kWave + lane];
      bl[i] = qb[(KS + i) * kWave + lane];
    }
    const uint16_t* seg = a.keys[s] + ((size_t)l * a.Hk + g) * (size_t)a.stride[s] * D;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(seg), (short)0, n * D * 2, 0x00020000);
    // chunk q = 64 i + lane of tile t: sample t 16 + q / CPR, chunk q mod CPR
    auto load = [&](int t, u32x4 (&V)[NI]) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int q = i * kWave + lane, u = t * kTile + q / CPR;
        const uint32_t off = (t < t1 && u < m)
                                 ? (uint32_t)sample_row(step, u) * (CPR * 16) + (q % CPR) * 16
                                 : 0x80000000u;
        V[i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kAuxNT);
      }
    };
    u32x4 V[NI];
    load(t0, V);
    for (int t = t0; t < t1; ++t) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int q = i * kWave + lane, R = q >> 4, C = q & 15;
        lt_[R * 16 + (C ^ (R & 15))] = V[i];
      }
      __builtin_amdgcn_wave_barrier();
      load(t + 1, V);
      u32x4 A[KS];
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
        A[i] = lt_[R * 16 + (C ^ (R & 15))];
      }
      __builtin_amdgcn_wave_barrier();
      const f32x4 acc = score_hilo<KS>(A, bh, bl);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int u = t * kTile + 4 * kg + j;
        if (colv && u < m) a.samp[(size_t)list * a.samp_stride + u] = acc[j] + 0.0f;
      }
    }
    T += t1 - t0;
  }
}

// Query prep and the sample pass in one launch (head-mode 0).  Block b works on
// one (stream, layer, KV head) group and kPsTiles of its sample tiles: it first
// forms the group's B tile exactly as k_prep does (the same sums in the same
// order, so every block of the group holds the same bits; the group's first
// block also writes them, and the column norms, for the streaming pass), keeps
// it in LDS, and then each wave gathers and scores its tiles as k_sample does.
// One launch instead of two: the sample no longer waits for a separate prep
// kernel to drain.
constexpr int kPsTiles = 32;   // sample tiles per block

struct PsArgs {
  int blk_base[kMaxStreams + 1];   // first block of each stream
  int spg[kMaxStreams];            // blocks per (layer, KV head) group of each stream
  int xcd_map;                     // block b plays (b mod 8) * (blocks / 8) + b / 8
};

template <int D>
__global__ __launch_bounds__(8 * D) void k_prep_sample(PrepArgs pa, ScoreArgs a, PsArgs ps) {
  constexpr int CPR = D / 8, TCH = 16 * CPR, NI = TCH / kWave, KS = D / 32;
  constexpr int NW = 8 * D / kWave;   // waves per block
  constexpr int PF = kPsTiles / NW;   // tiles per wave, all in flight
  union PsShared {
    float part[kPrepGroups][2 * D][8];
    u32x4 tiles[NW][TCH];
  };
  __shared__ PsShared sh;
  __shared__ u32x4 bsh[2 * KS * kWave];
  __shared__ float sout[kMaxGroup][kPsTiles * kTile];   // the block's scores, written out by whole lines
  int s = 0;
  // On a 256-CU device block b runs on XCD b mod 8: with xcd_map each XCD
  // takes a contiguous run of the group-major block order, so the slices of
  // a group mostly share one XCD and its L2 serves their query reads after
  // the first.
  const int vb = ps.xcd_map ? (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
  while (vb >= ps.blk_base[s + 1]) ++s;
  const int rem = vb - ps.blk_base[s];
  const int lg = rem / ps.spg[s], slice = rem - lg * ps.spg[s];
  const int l = lg / a.Hk, g = lg - l * a.Hk;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  const int n = a.n[s], m = a.units[s], nt = a.ntile[s];
  const int64_t step = a.samp_step[s];
  const uint16_t* seg = a.keys[s] + ((size_t)l * a.Hk + g) * (size_t)a.stride[s] * D;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(seg), (short)0, n * D * 2, 0x00020000);
  // wave w scores tiles slice kPsTiles + w + NW p (p < PF); chunk q = 64 i +
  // lane of tile t is chunk q mod CPR of sample t 16 + q / CPR; past the
  // group's tiles or samples the loads read zeros without touching memory.
  // The first tile's loads go out before the query prep (they need no B
  // tile), the others after it (all of them before would spill).
  u32x4 V[PF][NI];
  auto issue = [&](int p) {
    const int t = slice * kPsTiles + wave + NW * p;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * kWave + lane, u = t * kTile + q / CPR;
      const uint32_t off = (t < nt && u < m) ? (uint32_t)sample_row(step, u) * (CPR * 16) + (q % CPR) * 16
                                             : 0x80000000u;
      V[p][i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kAuxNT);
    }
  };
  issue(0);
  prep_b<D>(pa, s * a.L + l, g, sh.part, bsh, slice == 0);
  __syncthreads();   // the B tile is in LDS and the partial sums are read no more
  u32x4* lt_ = sh.tiles[wave];
  u32x4 bh[KS], bl[KS];
#pragma unroll
  for (int i = 0; i < KS; ++i) {
    bh[i] = bsh[i * kWave + lane];
    bl[i] = bsh[(KS + i) * kWave + lane];
  }
#pragma unroll
  for (int p = 1; p < PF; ++p) issue(p);
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    const int t = slice * kPsTiles + wave + NW * p;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * kWave + lane, R = q >> 4, C = q & 15;
      lt_[R * 16 + (C ^ (R & 15))] = V[p][i];
    }
    __builtin_amdgcn_wave_barrier();
    u32x4 A[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
      A[i] = lt_[R * 16 + (C ^ (R & 15))];
    }
    __builtin_amdgcn_wave_barrier();
    const f32x4 acc = score_hilo<KS>(A, bh, bl);
#pragma unroll
    for (int j = 0; j < 4; ++j) sout[col][(wave + NW * p) * kTile + 4 * kg + j] = acc[j] + 0.0f;
  }
  __syncthreads();
  // column c's kPsTiles * 16 scores are consecutive samples of list c of the
  // group: contiguous in the sample buffer
  const int u0 = slice * kPsTiles * kTile, nu = min(kPsTiles * kTile, m - u0);
  const int list0 = s * a.NL + l * a.Hq + g * a.G;
  for (int i = threadIdx.x; i < a.G * kPsTiles * kTile; i += blockDim.x) {
    const int c = i / (kPsTiles * kTile), u = i - c * (kPsTiles * kTile);
    if (u < nu) a.samp[(size_t)(list0 + c) * a.samp_stride + u0 + u] = sout[c][u];
  }
}

// Head mode 1, sample and exact-recompute roles: one layer per item; every
// tile's rows are read for each KV head in the MFMA A layout.
// One item (stream, layer, chunk of units) of k_score_hm with the layer's B
// operand b in registers.  Called by whole waves of a block.
template <int D, int KIND>
__device__ __forceinline__ void score_hm_item(const ScoreArgs& a, int s, int l, int u0, int u1, bool wr,
                                              const u32x4 (&b)[D / 32]) {
  constexpr int KS = D / 32;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  const bool colv = col == 0;
  const int list = s * a.NL + l;
  const size_t gstride = (size_t)a.stride[s] * D;
  const uint16_t* base = a.keys[s] + (size_t)l * a.Hk * gstride + 8 * kg;
  const int ntiles = (u1 - u0 + kTile - 1) / kTile;
  for (int t = wave; t < ntiles; t += nw) {
    const int u = u0 + t * kTile + rl;
    const bool ok = u < u1;
    const int64_t row = ok ? unit_row<KIND>(a, s, u) : 0;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    for (int g = 0; g < a.Hk; ++g) {
      const uint16_t* p = base + g * gstride + row * D;
      u32x4 A[KS];
#pragma unroll
      for (int i = 0; i < KS; ++i) A[i] = ok ? ld_nt(p + 32 * i) : u32x4{0, 0, 0, 0};
      hm_accumulate<KS>(A, b, g, v);
    }
    emit<KIND>(a, s, list, colv, wr, u0 + t * kTile, u1, hm_finish(v), kg);
  }
}

template <int D, int KIND>
__global__ __launch_bounds__(256) void k_score_hm(ScoreArgs a) {
  static_assert(KIND != K_STREAM, "head-mode-1 streaming runs in k_stream_hm");
  constexpr int KS = D / 32;
  const int lane = threadIdx.x & (kWave - 1), col = lane & 15;
  for (int item = blockIdx.x; item < a.total_items; item += gridDim.x) {
    int s = 0;
    while (item >= a.item_base[s + 1]) ++s;
    const int rem = item - a.item_base[s];
    const int units = a.units[s];
    const int nch = (units + a.chunk - 1) / a.chunk;
    const int chunk = rem % nch, l = rem / nch;
    const int u0 = chunk * a.chunk, u1 = min(units, u0 + a.chunk);
    bool wr = false;
    if (KIND == K_FULL) {
      wr = col == 0 && l == a.only_list;
      if (!__any(wr)) continue;
    }
    u32x4 b[KS];
    hm_load_b<KS>(a.qB + (size_t)(s * a.L + l) * a.Hk * (2 * KS * kWave), a.Hk, b);
    score_hm_item<D, KIND>(a, s, l, u0, u1, wr, b);
  }
}

// Head mode 1, the query prep fused into the sample pass (k_score_hm_prep),
// for batches whose query-head groups are small (G * n_q <= kHmPrepTerms):
// every item's block forms its layer's head-mean B columns itself, the same
// sums in k_prep's order (token groups j mod 4, heads outer, tokens inner, the
// four groups added in order; the column's L1 norm by the same butterfly);
// the block of the layer's first chunk also writes the B tiles and the column
// norms for the later kernels, which read the same bits as the sample.
// At the paper's settings (one query token) this takes a kernel and its
// boundary off the chain before the streaming pass.
constexpr int kHmPrepTerms = 64;

template <int D>
__device__ __forceinline__ void hm_prep_block(const PrepArgs& pa, int s, int l, int Hk, int G,
                                              u32x4 (*colB)[2][D / 32][4], float (*l1p)[16], bool publish) {
  constexpr int KS = D / 32, NE = D / 8;
  const int pair = s * pa.L + l;
  const uint16_t* q = pa.q[pair];
  const int nq = pa.nq[s];
  const float scale = pa.qscale[s];
  // thread (g, ec): dims 8 ec .. 8 ec + 7 of KV head g's column
  for (int c = threadIdx.x; c < Hk * NE; c += blockDim.x) {
    const int g = c / NE, ec = c - g * NE;
    float acc[4][8];
#pragma unroll
    for (int tg = 0; tg < 4; ++tg)
#pragma unroll
      for (int w = 0; w < 8; ++w) acc[tg][w] = 0.f;
#pragma unroll
    for (int tg = 0; tg < 4; ++tg) {
      for (int h = g * G; h < g * G + G; ++h) {
        for (int j = tg; j < nq; j += 4) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(q + ((size_t)h * nq + j) * D + 8 * ec);
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            acc[tg][2 * w] += bf16_lo(v[w]);
            acc[tg][2 * w + 1] += bf16_hi(v[w]);
          }
        }
      }
    }
    u32x4 hi, lo;
    float l1 = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float y0 = acc[0][2 * w], y1 = acc[0][2 * w + 1];
#pragma unroll
      for (int tg = 1; tg < 4; ++tg) { y0 += acc[tg][2 * w]; y1 += acc[tg][2 * w + 1]; }
      const float x0 = y0 * scale, x1 = y1 * scale;
      l1 += fabsf(x0) + fabsf(x1);
      const uint16_t a0 = bf16_rne(x0), a1 = bf16_rne(x1);
      const uint16_t b0 = bf16_rne(x0 - __uint_as_float((uint32_t)a0 << 16));
      const uint16_t b1 = bf16_rne(x1 - __uint_as_float((uint32_t)a1 << 16));
      hi[w] = (uint32_t)a0 | ((uint32_t)a1 << 16);
      lo[w] = (uint32_t)b0 | ((uint32_t)b1 << 16);
    }
    const int i = ec >> 2, kg = ec & 3;
    colB[g][0][i][kg] = hi;
    colB[g][1][i][kg] = lo;
    l1p[g][ec] = l1;
  }
  __syncthreads();
  if (!publish) return;
  // the whole B tiles (columns 1..15 zero, as k_prep leaves them in head mode 1)
  u32x4* out = pa.qB + (size_t)pair * Hk * (2 * KS * kWave);
  for (int e = threadIdx.x; e < Hk * 2 * KS * kWave; e += blockDim.x) {
    const int g = e / (2 * KS * kWave), r = e - g * (2 * KS * kWave);
    const int part = r / (KS * kWave), r2 = r - part * (KS * kWave), i = r2 / kWave, ln = r2 - i * kWave;
    out[e] = (ln & 15) == 0 ? colB[g][part][i][ln >> 4] : u32x4{0, 0, 0, 0};
  }
  // the column norm: k_prep's butterfly over the NE chunks (o = NE / 2 .. 1)
  if (pa.qcol)
    for (int e = threadIdx.x; e < Hk * 16; e += blockDim.x) {
      const int g = e >> 4, cl = e & 15;
      float nrm = 0.f;
      if (cl == 0) {
        float v[NE];
#pragma unroll
        for (int k = 0; k < NE; ++k) v[k] = l1p[g][k];
#pragma unroll
        for (int o = NE / 2; o > 0; o >>= 1) {
          float w[NE];
#pragma unroll
          for (int k = 0; k < NE; ++k) w[k] = v[k] + v[k ^ o];
#pragma unroll
          for (int k = 0; k < NE; ++k) v[k] = w[k];
        }
        nrm = v[0];
      }
      pa.qcol[((size_t)pair * Hk + g) * 16 + cl] = nrm;
    }
}

template <int D>
__global__ __launch_bounds__(256) void k_score_hm_prep(PrepArgs pa, ScoreArgs a) {
  constexpr int KS = D / 32;
  __shared__ u32x4 colB[8][2][KS][4];
  __shared__ float l1p[8][16];
  const int lane = threadIdx.x & (kWave - 1), c = lane & 15, kg = lane >> 4, g = c & 7;
  for (int item = blockIdx.x; item < a.total_items; item += gridDim.x) {
    int s = 0;
    while (item >= a.item_base[s + 1]) ++s;
    const int rem = item - a.item_base[s];
    const int units = a.units[s];
    const int nch = (units + a.chunk - 1) / a.chunk;
    const int chunk = rem % nch, l = rem / nch;
    const int u0 = chunk * a.chunk, u1 = min(units, u0 + a.chunk);
    __syncthreads();   // the previous item's B columns are read no more
    hm_prep_block<D>(pa, s, l, a.Hk, a.G, colB, l1p, chunk == 0);
    u32x4 b[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) b[i] = g < a.Hk ? colB[g][c < 8 ? 0 : 1][i][kg] : u32x4{0, 0, 0, 0};
    score_hm_item<D, K_SAMPLE>(a, s, l, u0, u1, false, b);
  }
}

// Head mode 1, streaming role: like k_stream, with the (stream, layer) lists
// as segments; a tile of 16 rows is read once per KV head (coalesced, through
// the wave's LDS tile), one sub-tile ahead.
template <int D>
__global__ __launch_bounds__(256) void k_stream_hm(ScoreArgs a) {
  constexpr int CPR = D / 8, TCH = 16 * CPR, NI = TCH / kWave, KS = D / 32;
  __shared__ u32x4 tiles[4][TCH];
  __shared__ uint64_t stage[4 * kStage];   // column 0 only
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  u32x4* lt_ = tiles[wave];
  uint64_t* st = stage + wave * kStage;
  const WaveRange wr = wave_range(a.tile_base[a.S], wave, a.sgroup, a.xcd_weights != 0);
  const int SW = wr.sw;
  for (int64_t T = wr.b0; T < wr.b1;) {
    int s = 0;
    while (T >= a.tile_base[s + 1]) ++s;
    const int64_t rem = T - a.tile_base[s];
    const int nt = a.ntile[s];
    const int l = (int)(rem / nt);
    const int tb = (int)(rem - (int64_t)l * nt);
    const int t1 = (int)min<int64_t>(nt, tb + (wr.b1 - T));
    const int t0 = first_tile(wr, T, tb);
    T += t1 - tb;
    if (t0 >= t1) continue;
    const int n = a.n[s], Hk = a.Hk;
    const bool colv = col == 0;
    const int list = s * a.NL + l;
    const float tau_f = ord_f32(colv ? a.tau[list] : 0xFFFFFFFFu);
    u32x4 b[KS];
    hm_load_b<KS>(a.qB + (size_t)(s * a.L + l) * Hk * (2 * KS * kWave), Hk, b);
    const uint16_t* lay = a.keys[s] + (size_t)l * Hk * a.stride[s] * D;
    // sub-tile (t, g): rows 16 t .. 16 t + 15 of KV head g, zeros past the list
    auto load = [&](int t, int g, u32x4 (&V)[NI]) {
      const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(lay + (size_t)g * a.stride[s] * D), (short)0, n * D * 2, 0x00020000);
      const uint32_t off = t < t1 ? (uint32_t)t * (TCH * 16) + lane * 16 : 0x80000000u;
#pragma unroll
      for (int i = 0; i < NI; ++i) V[i] = __builtin_amdgcn_raw_buffer_load_b128(r, off + i * kWave * 16, 0, kAuxNT);
    };
    u32x4 V[NI];
    load(t0, 0, V);
    int lc = 0;
    for (int t = t0; t < t1; t += SW) {
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      for (int g = 0; g < Hk; ++g) {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const int q = i * kWave + lane, R = q >> 4, C = q & 15;
          lt_[R * 16 + (C ^ (R & 15))] = V[i];
        }
        __builtin_amdgcn_wave_barrier();
        if (g + 1 < Hk) load(t, g + 1, V);
        else load(t + SW, 0, V);
        u32x4 A[KS];
#pragma unroll
        for (int i = 0; i < KS; ++i) {
          const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
          A[i] = lt_[R * 16 + (C ^ (R & 15))];
        }
        __builtin_amdgcn_wave_barrier();
        hm_accumulate<KS>(A, b, g, v);
      }
      double unused = 0.0;
      stream_emit(a, list, colv, col, tau_f, t * kTile, n, hm_finish(v), kg, st, lc, unused, false);
    }
    if (__any(lc > 0)) stage_flush(a, list, colv, col, kg, st, lc);
  }
}

// Streaming pass, head mode 1 with attention probabilities.  Like k_stream_hm,
// the segments are (stream, layer) lists and a 16-row tile is read once per KV
// head; but each head keeps its own logits: the B tiles are head mode 0's (hi
// and lo, the G query heads of a KV head in the columns), all HK of them in
// registers for the visit.  Lane (c, kg) turns the logits of head g G + c into
// e = exp(s - Lhat) (the sample estimate of the head's log-sum-exp), the
// row's 16 columns and HK heads are summed in a fixed butterfly, and
// alpha_hat = that sum / H_q.  Rows with alpha_hat >= tau_hat are staged as
// candidates; every other row adds e / (H_q tau_hat), below 1 for it, to its
// head's fixed-point sum.  MFMA work per key vector is that of head mode 0.
template <int D, int HK>
__global__ __launch_bounds__(256) void k_stream_hp(ScoreArgs a) {
  constexpr int CPR = D / 8, TCH = 16 * CPR, NI = TCH / kWave, KS = D / 32;
  __shared__ u32x4 tiles[4][TCH];
  __shared__ uint64_t stage[4 * kStage];   // column 0 only
  __shared__ unsigned long long fl_below[kHpHeads];   // the block's fixed-point sums per head
  __shared__ uint32_t fl_lmax;
  for (int h = threadIdx.x; h < kHpHeads; h += blockDim.x) fl_below[h] = 0;
  if (threadIdx.x == 0) fl_lmax = 0;
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  u32x4* lt_ = tiles[wave];
  uint64_t* st = stage + wave * kStage;
  const WaveRange wr = wave_range(a.tile_base[a.S], wave, a.sgroup, a.xcd_weights != 0);
  const int SW = wr.sw;
  const float inv_h = 1.0f / (float)a.Hq;
  for (int64_t T = wr.b0; T < wr.b1;) {
    int s = 0;
    while (T >= a.tile_base[s + 1]) ++s;
    const int64_t rem = T - a.tile_base[s];
    const int nt = a.ntile[s];
    const int l = (int)(rem / nt);
    const int tb = (int)(rem - (int64_t)l * nt);
    const int t1 = (int)min<int64_t>(nt, tb + (wr.b1 - T));
    const int t0 = first_tile(wr, T, tb);
    T += t1 - tb;
    // (every wave of the block takes part in the segment's sums, with or
    // without tiles of its own)
    const int n = a.n[s];
    const bool colv = col == 0;
    const int list = s * a.NL + l;
    const float tau_all = ord_f32(a.tau[list]);
    const float tau_f = colv ? tau_all : __uint_as_float(0x7FC00000u);   // staging lanes only
    const double bscale = tau_all > 0.f ? 1.0 / ((double)a.Hq * (double)tau_all) : 0.0;
    const size_t hb = (size_t)(s * a.L + l) * a.Hq;   // head 0 of the layer
    u32x4 bh[HK][KS], bl[HK][KS];
    float lh[HK];
#pragma unroll
    for (int g = 0; g < HK; ++g) {
      const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * HK + g) * (2 * KS * kWave);
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        bh[g][i] = qb[i * kWave + lane];
        bl[g][i] = qb[(KS + i) * kWave + lane];
      }
      lh[g] = col < a.G ? a.lhat[hb + g * a.G + col] : INFINITY;   // exp(s - inf) = 0 in padding columns
    }
    const uint16_t* lay = a.keys[s] + (size_t)l * HK * a.stride[s] * D;
    auto load = [&](int t, int g, u32x4 (&V)[NI]) {
      const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(lay + (size_t)g * a.stride[s] * D), (short)0, n * D * 2, 0x00020000);
      const uint32_t off = t < t1 ? (uint32_t)t * (TCH * 16) + lane * 16 : 0x80000000u;
#pragma unroll
      for (int i = 0; i < NI; ++i) V[i] = __builtin_amdgcn_raw_buffer_load_b128(r, off + i * kWave * 16, 0, kAuxNT);
    };
    u32x4 V[NI];
    load(t0, 0, V);
    int lc = 0;
    uint32_t lmax = 0;   // largest alpha_hat left out (ordered bits; 0 below every value)
    double bsum[HK];
#pragma unroll
    for (int g = 0; g < HK; ++g) bsum[g] = 0.0;
    for (int t = t0; t < t1; t += SW) {
      float e[HK][4];
      f32x4 rs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int g = 0; g < HK; ++g) {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          const int q = i * kWave + lane, R = q >> 4, C = q & 15;
          lt_[R * 16 + (C ^ (R & 15))] = V[i];
        }
        __builtin_amdgcn_wave_barrier();
        if (g + 1 < HK) load(t, g + 1, V);
        else load(t + SW, 0, V);
        u32x4 A[KS];
#pragma unroll
        for (int i = 0; i < KS; ++i) {
          const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
          A[i] = lt_[R * 16 + (C ^ (R & 15))];
        }
        __builtin_amdgcn_wave_barrier();
        const f32x4 acc = score_hilo<KS>(A, bh[g], bl[g]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          e[g][j] = __expf(acc[j] - lh[g]);
          rs[j] += e[g][j];
        }
      }
      rs = hm_finish(rs);   // every lane of a 16-lane row: the sum over its 16 columns
      f32x4 al;
#pragma unroll
      for (int j = 0; j < 4; ++j) al[j] = rs[j] * inv_h + 0.0f;
      double unused = 0.0;
      stream_emit(a, list, colv, col, tau_f, t * kTile, n, al, kg, st, lc, unused, false);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (t * kTile + 4 * kg + j < n && !(al[j] >= tau_all)) {
          lmax = max(lmax, ord_u32(al[j]));
#pragma unroll
          for (int g = 0; g < HK; ++g) bsum[g] += (double)e[g][j];
        }
      }
    }
    if (__any(lc > 0)) stage_flush(a, list, colv, col, kg, st, lc);
    // The waves of a group end a segment together: each wave rounds its
    // per-head sums to fixed point as below_flush does, the block adds the
    // integers in LDS and makes one atomic per head (and one for the
    // largest estimate left out), not one per wave.
#pragma unroll
    for (int g = 0; g < HK; ++g) {
      double x = bsum[g];
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      if (kg == 0 && col < a.G && x > 0.0)
        atomicAdd(&fl_below[g * a.G + col], (unsigned long long)llrint(ldexp(x * bscale, kBelowExp)));
    }
    for (int o = 32; o > 0; o >>= 1) lmax = max(lmax, (uint32_t)__shfl_xor((int)lmax, o));
    if (lane == 0 && lmax > 0) atomicMax(&fl_lmax, lmax);
    __syncthreads();
    if (wave == 0) {
      for (int h = lane; h < a.Hq; h += kWave) {
        const unsigned long long b = fl_below[h];
        if (b) atomicAdd(reinterpret_cast<unsigned long long*>(&a.below[hb + h]), b);
        fl_below[h] = 0;
      }
      if (lane == 0) {
        if (fl_lmax > 0) atomicMax(&a.left_max[list], fl_lmax);
        fl_lmax = 0;
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Wave and block reductions (DPP within rows of 16 lanes, then readlane)
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false));  // row_ror 4
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false));  // row_ror 8
  const uint32_t a = __builtin_amdgcn_readlane(v, 15), b = __builtin_amdgcn_readlane(v, 31);
  const uint32_t c = __builtin_amdgcn_readlane(v, 47), d = __builtin_amdgcn_readlane(v, 63);
  return max(max(a, b), max(c, d));
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) { return ~wave_max_u32(~v); }

// Block min and max; `sh` holds 2 * (blockDim/64) words.
__device__ void block_minmax_u32(uint32_t& mn, uint32_t& mx, uint32_t* sh) {
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  mn = wave_min_u32(mn);
  mx = wave_max_u32(mx);
  if ((threadIdx.x & (kWave - 1)) == 0) { sh[2 * w] = mn; sh[2 * w + 1] = mx; }
  __syncthreads();
  for (int i = 0; i < nw; ++i) { mn = min(mn, sh[2 * i]); mx = max(mx, sh[2 * i + 1]); }
  __syncthreads();
}

// Exact r-th largest (1 <= r <= #valid) of the values the block holds in
// registers, all in [lo, hi]: radix selection over the value range, 8 bits of
// (v - lo) per round, so about three rounds for scores of one sign and exponent
// band.  WIDE: the first round takes 11 bits (2048 bins spread the bulk of many
// values, which keeps same-bin LDS atomics rare, and saves a round).  Returns
// the value; `n_greater` and `n_equal` count the valid values above it and
// equal to it.  `hist` holds 512 words, kSelHist when WIDE (the wide
// histogram padded by pad32).
constexpr int kSelHist = 2048 + 64 + 512;

// Ends a radix selection whose current bin [lo, hi] holds eq <= 64 values: they
// are gathered into `vals` (64 words, no longer read as a histogram) and wave 0
// ranks them by counting; the need-th largest t of the bin gives lo = hi = t,
// need = its rank among the values equal to t, eq = their count.  res[3] is the
// gather counter; res[0..2] carry the result.  Called by the whole block.
template <int N>
__device__ void finish_bin_by_counting(const uint32_t (&v)[N], const bool (&ok)[N], uint32_t& lo,
                                       uint32_t& hi, uint32_t& need, uint32_t& eq, uint32_t* vals,
                                       uint32_t* res) {
  if (threadIdx.x == 0) res[3] = 0;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < N; ++i)
    if (ok[i] && v[i] >= lo && v[i] <= hi) {
      const uint32_t slot = atomicAdd(&res[3], 1u);
      if (slot < (uint32_t)kWave) vals[slot] = v[i];   // the bin holds eq <= 64 values
    }
  __syncthreads();
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const uint32_t mine = lane < (int)eq ? vals[lane] : 0u;
    uint32_t gt = 0, ge = 0;
    // the other values from the lanes' registers (j is uniform)
#pragma unroll 8
    for (uint32_t j = 0; j < eq; ++j) {
      const uint32_t o = (uint32_t)__builtin_amdgcn_readlane((int)mine, (int)j);
      gt += o > mine;
      ge += o >= mine;
    }
    // t: fewer than need values of the bin above it, at least need at or above it
    const uint64_t hit = __ballot(lane < (int)eq && gt < need && need <= ge);
    if (lane == __builtin_ctzll(hit)) { res[0] = mine; res[1] = gt; res[2] = ge - gt; }
  }
  __syncthreads();
  lo = hi = res[0];
  need -= res[1];
  eq = res[2];
}

template <int N, bool WIDE>
__device__ uint32_t block_select_range(const uint32_t (&v)[N], const bool (&ok)[N], uint32_t lo,
                                       uint32_t hi, uint32_t r, uint32_t* hist, uint32_t* res,
                                       uint32_t& n_greater, uint32_t& n_equal) {
  uint32_t* wide = hist + 512;
  for (int i = threadIdx.x; i < (WIDE ? kSelHist : 512); i += blockDim.x) hist[i] = 0;
  uint32_t need = r, eq = 0;
  bool rounds = false;
  int buf = 0;
  __syncthreads();
  if (WIDE && lo < hi) {   // first round: 11 bits
    const uint32_t span = hi - lo;
    const int bits = 32 - __clz(span);
    const int shift = bits > 11 ? bits - 11 : 0;
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (ok[i] && v[i] >= lo && v[i] <= hi) atomicAdd(&wide[pad32((v[i] - lo) >> shift)], 1u);
    __syncthreads();
    find_digit_wide<32, true>(wide, need, res);
    need -= res[1];
    eq = res[2];
    lo += res[0] << shift;
    hi = (uint32_t)min((uint64_t)hi, (uint64_t)lo + (((uint64_t)1 << shift) - 1));
    rounds = true;
    // a bin of at most 64 values (the usual case for a cut in the tail of a
    // sample) is ranked by counting instead of further radix rounds
    if (lo < hi && eq <= (uint32_t)kWave) finish_bin_by_counting<N>(v, ok, lo, hi, need, eq, wide, res);
  }
  while (lo < hi) {
    const uint32_t span = hi - lo;
    const int bits = 32 - __clz(span);              // span < 2^bits
    const int shift = bits > 8 ? bits - 8 : 0;
    uint32_t* h = hist + buf * 256;
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (ok[i] && v[i] >= lo && v[i] <= hi) atomicAdd(&h[(v[i] - lo) >> shift], 1u);
    __syncthreads();
    for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[(buf ^ 1) * 256 + i] = 0;
    find_digit(h, need, res);                        // ends with a barrier
    need -= res[1];
    eq = res[2];
    lo += res[0] << shift;
    hi = (uint32_t)min((uint64_t)hi, (uint64_t)lo + (((uint64_t)1 << shift) - 1));
    rounds = true;
    // this round's histogram is read no more: it takes the values of a small bin
    if (lo < hi && eq <= (uint32_t)kWave) finish_bin_by_counting<N>(v, ok, lo, hi, need, eq, h, res);
    buf ^= 1;
  }
  if (!rounds) {  // every valid value equals lo
    uint32_t c = 0;
#pragma unroll
    for (int i = 0; i < N; ++i) c += ok[i];
    if (threadIdx.x == 0) hist[0] = 0;
    __syncthreads();
    atomicAdd(&hist[0], c);
    __syncthreads();
    eq = hist[0];
    __syncthreads();
  }
  n_greater = r - need;
  n_equal = eq;
  return lo;
}

// ---------------------------------------------------------------------------
// k_thresh: per list, the r-th largest sample score as an ordered uint32
// ---------------------------------------------------------------------------
struct ListArgs {
  int NL, S, cap, k_max, top_k, hist_f;
  int score_mode;                          // 1: attention probabilities
  int hm_prob;                             // head mode 1 with attention probabilities
  int NLs;                                 // sampled lists per stream (L * H_q when hm_prob)
  uint64_t* below;                         // score_mode 1: fixed-point exp sums below each cut-off
  float* lhat;                             // hm_prob: sample log-sum-exp estimate of each (layer, head)
  float* cand_sc;                          // hm_prob: [S*NL][H_q][cap] per-head candidate logits
  float* cand_lse;                         // hm_prob: [S*NL][H_q] exact log-sum-exp of each head's list
  uint32_t* left_max;                      // hm_prob: [S*NL] largest alpha_hat left out (ordered bits)
  int32_t m[kMaxStreams], r[kMaxStreams], kk[kMaxStreams], n[kMaxStreams];
  int32_t f[kMaxStreams], rpf[kMaxStreams];
  const int32_t* frame_off[kMaxStreams];   // from the first candidate frame; values are absolute rows
  int64_t row0[kMaxStreams];               // the first candidate row
  const float* samp;
  int samp_stride;
  uint32_t* tau;
  uint32_t* cnt;
  uint64_t* cand;                          // candidate keys (rewritten with exact values in hm_prob)
  // per-frame votes and fixed-point attention mass of each stream (window-relative frames)
  int f_max;
  int32_t* votes_g;    // [S][f_max]
  int64_t* massfx_g;   // [S][f_max] score sums at scale 2^sexp[s]
  int32_t* sexp;       // [S]
  const float* qcol;   // [S][L][H_kv][16] query column L1 norms
  const uint32_t* kmax[kMaxStreams];   // the index's largest |key element| (float bits)
  // exact fallback: the list's scores are recomputed from the keys
  int L, Hq, Hk, G, head_mode;
  const uint16_t* keys[kMaxStreams];
  int32_t stride[kMaxStreams];
  const u32x4* qB;
  int32_t* dbg_pos;
  float* dbg_score;
  int32_t* dbg_stats;
  uint32_t* dyn_ctr;   // the streaming pass's chunk counters (zeroed by k_thresh)
};

__device__ __forceinline__ int frame_of_row(const ListArgs& a, int s, uint32_t row) {
  if (a.rpf[s] > 0) return (int)(row / (uint32_t)a.rpf[s]);
  const int32_t* off = a.frame_off[s];
  const int64_t r = (int64_t)row + a.row0[s];
  int lo = 0, hi = a.f[s] - 1;  // largest f with off[f] <= row
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)off[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Fixed-point exponent of a stream's attention mass.  A score is a dot product
// of a scaled query column with a key row, so |score| <= |q|_1 * max|K| (head
// mode 1 sums the KV heads' columns); with 2% headroom for fp32 rounding this
// bounds all E = NL * kk selected scores of the stream, and at scale 2^x with
// x = 61 - e - c (bound < 2^e, E <= 2^c) any sum of them stays below 2^61.
// Computed by every lane of wave 0 (no block barrier); every selection block
// of the stream gets the same value.
__device__ int stream_exponent(const ListArgs& a, int s) {
  // attention probabilities: a list's selected values add up to at most 1, so
  // a frame's mass is below NL <= 2^12 and 2^50 keeps every sum below 2^62
  if (a.score_mode == 1) return kProbMassExp;
  const int L = a.L, Hk = a.Hk;
  const float* qc = a.qcol + (size_t)s * L * Hk * 16;
  const float km = __uint_as_float(*a.kmax[s]);   // issued with the column loads
  float b = 0.f;
  if (a.head_mode == 0) {
#pragma unroll 4
    for (int i = threadIdx.x; i < L * Hk * 16; i += kWave) b = fmaxf(b, qc[i]);
  } else {
    for (int l = threadIdx.x; l < L; l += kWave) {
      float t = 0.f;
      for (int g = 0; g < Hk; ++g) t += qc[(l * Hk + g) * 16];
      b = fmaxf(b, t);
    }
  }
  b = __uint_as_float(wave_max_u32(__float_as_uint(b)));   // non-negative: ordered as integers
  const float bound = b * km * 1.02f;
  const int E = a.NL * a.kk[s];
  int x = 120;                          // all scores are zero
  if (!(bound <= 3.0e38f)) {
    x = -120;                           // non-finite keys or queries
  } else if (bound > 0.f) {
    int e;
    frexpf(bound, &e);                  // bound < 2^e
    const int c = (E > 1) ? 32 - __clz(E - 1) : 0;
    x = min(120, max(-120, 61 - e - c));
  }
  return x;
}

// The stream's mass exponent in the selection block (LDS).
__device__ __forceinline__ int& list_mass_exponent() {
  __shared__ int xs;
  return xs;
}

// The sample (m <= N * 1024 scores, N <= kThrItems, chosen at launch from the
// largest sample) sits in registers.  The blocks of a stream also clear its
// frame accumulators.
template <int N>
__device__ __forceinline__ void thresh_list(const ListArgs& a) {
  __shared__ uint32_t hist[kSelHist];
  __shared__ uint32_t res[4];
  __shared__ uint32_t mm[32];
  const int list = blockIdx.x, s = list / a.NL, ll = list - s * a.NL;
  const int m = a.m[s], r = a.r[s];
  if (threadIdx.x == 0) a.cnt[list] = 0;
  if (a.below && !a.hm_prob && threadIdx.x == 0) a.below[list] = 0;   // hm_prob: per head, in k_lhat
  if (list == 0 && threadIdx.x < kDynCtr) a.dyn_ctr[threadIdx.x * kDynStride] = 0;
  {
    int32_t* vg = a.votes_g + (size_t)s * a.f_max;
    int64_t* mg = a.massfx_g + (size_t)s * a.f_max;
    for (int f = ll * 1024 + threadIdx.x; f < a.f[s]; f += a.NL * 1024) {
      vg[f] = 0;
      mg[f] = 0;
    }
  }
  if (m == 0 || r == 0) {
    if (threadIdx.x == 0) a.tau[list] = 0xFFFFFFFFu;
    return;
  }
  const float* v = a.samp + (size_t)list * a.samp_stride;
  uint32_t x[N];
  bool ok[N];
  uint32_t mn = 0xFFFFFFFFu, mx = 0;
  // every load issued at once, from clamped in-bounds indices (m >= 1)
#pragma unroll
  for (int it = 0; it < N; ++it) x[it] = __float_as_uint(v[min((int)threadIdx.x + it * 1024, m - 1)]);
#pragma unroll
  for (int it = 0; it < N; ++it) {
    ok[it] = (int)threadIdx.x + it * 1024 < m;
    x[it] = ok[it] ? ord_u32(__uint_as_float(x[it]) + 0.0f) : 0u;
    if (ok[it]) { mn = min(mn, x[it]); mx = max(mx, x[it]); }
  }
  block_minmax_u32(mn, mx, mm);
  uint32_t ng, ne;
  const uint32_t t = block_select_range<N, true>(x, ok, mn, mx, (uint32_t)r, hist, res, ng, ne);
  if (threadIdx.x == 0) a.tau[list] = t;
}

// One block per list.  With up to two lists per CU the kernel takes the
// registers it wants (90 VGPRs: one block per CU); with more lists (the
// 16-stream batch: 1,536) the dense variant fits two blocks per CU in 64 VGPRs
// with a few spills, three rounds of blocks instead of six (41 -> 32 us on that
// batch).
template <int N>
__global__ __launch_bounds__(1024) void k_thresh(ListArgs a) {
  thresh_list<N>(a);
}
template <int N>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8, 8))) void k_thresh_dense(ListArgs a) {
  thresh_list<N>(a);
}

// k_prep_thresh: query prep, sample scores and the cut-off of one list per
// block in a single launch (head mode 0, d = 128, when every list's block fits
// one round and the sample fits N slots per thread; used for short samples).  The block forms its list
// group's B tile with the prep's exact sums (the group's first list publishes
// it for the streaming pass), scores every sampled row of the group against it
// with the sample pass's arithmetic (so a row gets the streaming pass's bits),
// keeps its own column in LDS and takes the r-th largest by the cut-off
// kernel's radix selection: the sample never goes through global memory and
// the cut-off needs no second launch.  The group's blocks read the same sampled
// rows; on a 256-CU device (block b on XCD b mod 8) each XCD takes whole list
// groups, so those rows come from its L2 after the first read.
struct PtArgs {
  int NL, L, Hq, Hk, G, f_max;
  int xcd_map;                          // lists (b mod 8) * (lists / 8) + b / 8
  const uint16_t* keys[kMaxStreams];
  int32_t stride[kMaxStreams];          // rows per (layer, KV head) in the arena
  int32_t n[kMaxStreams];               // candidate rows
  int32_t m[kMaxStreams];               // sampled rows per list group
  int32_t r[kMaxStreams];               // rank of the cut-off in the sample
  int32_t f[kMaxStreams];               // candidate frames
  int64_t samp_step[kMaxStreams];
  uint32_t* tau;
  uint32_t* cnt;
  uint64_t* below;                      // score mode 1, else null
  uint32_t* dyn_ctr;
  int32_t* votes_g;
  int64_t* massfx_g;
};

constexpr int kPtDepth = 2;   // sample tiles in flight per wave

template <int N>
__global__ __launch_bounds__(1024) void k_prep_thresh(PrepArgs pa, PtArgs a) {
  constexpr int D = 128, CPR = D / 8, TCH = 16 * CPR, NI = TCH / kWave, KS = D / 32, NW = 1024 / kWave;
  union PtShared {
    float part[kPrepGroups][2 * D][8];
    u32x4 tiles[NW][TCH];
  };
  __shared__ PtShared sh;
  __shared__ u32x4 bsh[2 * KS * kWave];
  __shared__ float sv[N * 1024];
  __shared__ uint32_t hist[kSelHist];
  __shared__ uint32_t res[4];
  __shared__ uint32_t mm[32];
  const int list = a.xcd_map ? (int)(blockIdx.x % 8) * (int)(gridDim.x / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
  const int s = list / a.NL, ll = list - s * a.NL;
  const int l = ll / a.Hq, h = ll - l * a.Hq, g = h / a.G, mycol = h - g * a.G;
  const int m = a.m[s], r = a.r[s];
  // the list's candidate count and exp sum, the streaming pass's chunk
  // counters and a slice of the stream's frame accumulators start at zero
  if (threadIdx.x == 0) a.cnt[list] = 0;
  if (a.below && threadIdx.x == 0) a.below[list] = 0;
  if (list == 0 && threadIdx.x < kDynCtr) a.dyn_ctr[threadIdx.x * kDynStride] = 0;
  {
    int32_t* vg = a.votes_g + (size_t)s * a.f_max;
    int64_t* mg = a.massfx_g + (size_t)s * a.f_max;
    for (int f = ll * 1024 + threadIdx.x; f < a.f[s]; f += a.NL * 1024) {
      vg[f] = 0;
      mg[f] = 0;
    }
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  const int n = a.n[s], nt = (m + kTile - 1) / kTile;
  const int64_t step = a.samp_step[s];
  const uint16_t* seg = a.keys[s] + ((size_t)l * a.Hk + g) * (size_t)a.stride[s] * D;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(seg), (short)0, n * D * 2, 0x00020000);
  // chunk q = 64 i + lane of tile t is chunk q mod CPR of sample t 16 + q / CPR;
  // past the samples the loads read zeros without touching memory
  auto issue = [&](int t, u32x4 (&V)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * kWave + lane, u = t * kTile + q / CPR;
      const uint32_t off = (t < nt && u < m) ? (uint32_t)sample_row(step, u) * (CPR * 16) + (q % CPR) * 16
                                             : 0x80000000u;
      V[i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kAuxNT);
    }
  };
  // wave w scores tiles w, w + NW, ...; kPtDepth of them in flight, the
  // first issued before the query prep (it needs no B tile), so that its
  // round trip overlaps the prep's
  u32x4 V[kPtDepth][NI];
  issue(wave, V[0]);
  prep_b<D>(pa, s * a.L + l, g, sh.part, bsh, mycol == 0);
#pragma unroll
  for (int d = 1; d < kPtDepth; ++d) issue(wave + d * NW, V[d]);
  if (m == 0 || r == 0) {
    if (threadIdx.x == 0) a.tau[list] = 0xFFFFFFFFu;
    return;
  }
  __syncthreads();   // the B tile is in LDS and the partial sums are read no more
  u32x4 bh[KS], bl[KS];
#pragma unroll
  for (int i = 0; i < KS; ++i) {
    bh[i] = bsh[i * kWave + lane];
    bl[i] = bsh[(KS + i) * kWave + lane];
  }
  u32x4* lt_ = sh.tiles[wave];
  for (int t0 = wave; t0 < nt; t0 += kPtDepth * NW) {
#pragma unroll
    for (int d = 0; d < kPtDepth; ++d) {
      const int t = t0 + d * NW;
      if (t >= nt) break;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int q = i * kWave + lane, R = q >> 4, C = q & 15;
        lt_[R * 16 + (C ^ (R & 15))] = V[d][i];
      }
      issue(t + kPtDepth * NW, V[d]);
      __builtin_amdgcn_wave_barrier();
      u32x4 A[KS];
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        const int q = rl * CPR + 4 * i + kg, R = q >> 4, C = q & 15;
        A[i] = lt_[R * 16 + (C ^ (R & 15))];
      }
      __builtin_amdgcn_wave_barrier();
      const f32x4 acc = score_hilo<KS>(A, bh, bl);
      if (col == mycol) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int u = t * kTile + 4 * kg + j;
          if (u < m) sv[u] = acc[j] + 0.0f;
        }
      }
    }
  }
  __syncthreads();
  uint32_t x[N];
  bool ok[N];
  uint32_t mn = 0xFFFFFFFFu, mx = 0;
#pragma unroll
  for (int it = 0; it < N; ++it) {
    const int i = (int)threadIdx.x + it * 1024;
    ok[it] = i < m;
    x[it] = ok[it] ? ord_u32(sv[i]) : 0u;
    if (ok[it]) { mn = min(mn, x[it]); mx = max(mx, x[it]); }
  }
  block_minmax_u32(mn, mx, mm);
  uint32_t ng, ne;
  const uint32_t t = block_select_range<N, true>(x, ok, mn, mx, (uint32_t)r, hist, res, ng, ne);
  if (threadIdx.x == 0) a.tau[list] = t;
}

// Launches the cut-off kernel with the fewest sample slots per thread that
// hold the largest sample.
void launch_thresh(const ListArgs& la, int lists, int m_max, bool dense, hipStream_t st) {
  const dim3 g(lists), b(1024);
  if (m_max <= 4096) {
    if (dense) hipLaunchKernelGGL(k_thresh_dense<4>, g, b, 0, st, la);
    else hipLaunchKernelGGL(k_thresh<4>, g, b, 0, st, la);
  } else if (m_max <= 8192) {
    if (dense) hipLaunchKernelGGL(k_thresh_dense<8>, g, b, 0, st, la);
    else hipLaunchKernelGGL(k_thresh<8>, g, b, 0, st, la);
  } else {
    if (dense) hipLaunchKernelGGL(k_thresh_dense<kThrItems>, g, b, 0, st, la);
    else hipLaunchKernelGGL(k_thresh<kThrItems>, g, b, 0, st, la);
  }
}

// Sum of a wave's doubles in a fixed butterfly (every lane gets the total).
__device__ __forceinline__ double wave_sum_f64(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max_f32(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

constexpr int kMaxHeadsHp = 128;   // query heads of a layer in head mode 1 (H_kv <= 8, G <= 16)

// Head mode 1 with attention probabilities: the cut-off of a layer's list
// comes from its sample in three launches.  k_lhat (one block per (list,
// head)) estimates the head's log-sum-exp over the list, Lhat_h =
// max + log(sum exp(s_h - max)) + log(n / m) over the head's sampled logits
// (block reductions in a fixed order), and clears the head's exp sum below
// the cut-off and the list's largest left-out estimate; k_alpha (one thread
// per sampled row) forms the row's estimated attention alpha_hat =
// mean_h exp(s_h - Lhat_h); k_thresh then takes the r-th largest alpha_hat
// as the cut-off tau_hat, as it does for logits.  The streaming pass keeps the
// rows with alpha_hat >= tau_hat, and k_select_hp proves from the exact
// normalisers that no other row can reach the top k (else it recomputes the
// list).
__global__ __launch_bounds__(1024) void k_lhat(ListArgs a) {
  __shared__ float redf[16];
  __shared__ double redd[16];
  const int list = blockIdx.x / a.Hq, h = blockIdx.x - list * a.Hq;
  const int s = list / a.NL, l = list - s * a.NL;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const size_t hb = (size_t)s * a.NLs + (size_t)l * a.Hq + h;   // the head's sampled list
  if (threadIdx.x == 0) {
    a.below[hb] = 0;
    if (h == 0) a.left_max[list] = 0;
  }
  const int m = a.m[s];
  if (m == 0) return;
  const float* v = a.samp + hb * a.samp_stride;
  float x[kThrItems];   // the sample (at most 16,384 rows) in registers, all loads in flight
#pragma unroll
  for (int it = 0; it < kThrItems; ++it) {
    const int u = (int)threadIdx.x + it * 1024;
    x[it] = u < m ? v[u] : -INFINITY;
  }
  float mx = -INFINITY;
#pragma unroll
  for (int it = 0; it < kThrItems; ++it) mx = fmaxf(mx, x[it]);
  mx = wave_max_f32(mx);
  if (lane == 0) redf[wave] = mx;
  __syncthreads();
  float M = redf[0];
  for (int w = 1; w < 16; ++w) M = fmaxf(M, redf[w]);
  double sm = 0.0;
#pragma unroll
  for (int it = 0; it < kThrItems; ++it)
    if ((int)threadIdx.x + it * 1024 < m) sm += (double)__expf(x[it] - M);
  sm = wave_sum_f64(sm);
  if (lane == 0) redd[wave] = sm;
  __syncthreads();
  if (threadIdx.x == 0) {
    double z = 0.0;
    for (int w = 0; w < 16; ++w) z += redd[w];
    a.lhat[hb] = M + (float)log(z) + logf((float)a.n[s] / (float)m);
  }
}

__global__ __launch_bounds__(256) void k_alpha(ListArgs a, float* alpha) {
  const int list = blockIdx.x, s = list / a.NL, l = list - s * a.NL;
  const int u = blockIdx.y * blockDim.x + threadIdx.x;
  if (u >= a.m[s]) return;
  const size_t hb = (size_t)s * a.NLs + (size_t)l * a.Hq;
  const float* v = a.samp + hb * a.samp_stride + u;
  float al = 0.f;
#pragma unroll 8
  for (int h = 0; h < a.Hq; ++h) al += __expf(v[(size_t)h * a.samp_stride] - a.lhat[hb + h]);
  alpha[(size_t)list * a.samp_stride + u] = al * (1.0f / (float)a.Hq) + 0.0f;
}

// Head mode 1, attention probabilities: every candidate's per-head logits with
// the streaming pass's arithmetic, 16 candidates per wave (each KV head's rows
// against head mode 0's B tiles, every head's key loads in flight at once),
// into cand_sc [list][head][cap]; lists that take the exact fallback are
// skipped.
template <int D, int HK>
__global__ __launch_bounds__(256) void k_cand_logits(ListArgs a) {
  constexpr int KS = D / 32;
  const int list = blockIdx.x, s = list / a.NL, l = list - s * a.NL;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const int kg = lane >> 4, rl = lane & 15, col = lane & 15;
  const uint32_t c = a.cnt[list];
  if (c < (uint32_t)a.kk[s] || c > (uint32_t)a.cap) return;
  const int n = (int)c, i0 = (blockIdx.y * (blockDim.x / kWave) + wave) * kTile;
  if (i0 >= n) return;   // uniform per wave
  const int G = a.G;
  const uint64_t* src = a.cand + (size_t)list * a.cap;
  float* cs = a.cand_sc + (size_t)list * a.Hq * a.cap;
  const size_t gstride = (size_t)a.stride[s] * D;
  const int i = i0 + rl;
  const uint32_t row = i < n ? key_row(src[i]) : 0u;
  u32x4 A[HK][KS];
#pragma unroll
  for (int g = 0; g < HK; ++g) {
    const uint16_t* p = a.keys[s] + ((size_t)l * HK + g) * gstride + (size_t)row * D + 8 * kg;
#pragma unroll
    for (int ii = 0; ii < KS; ++ii) A[g][ii] = i < n ? ld_nt(p + 32 * ii) : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int g = 0; g < HK; ++g) {
    const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * HK + g) * (2 * KS * kWave);
    u32x4 bh[KS], bl[KS];
#pragma unroll
    for (int ii = 0; ii < KS; ++ii) {
      bh[ii] = qb[ii * kWave + lane];
      bl[ii] = qb[(KS + ii) * kWave + lane];
    }
    const f32x4 acc = score_hilo<KS>(A[g], bh, bl);
    if (col < G) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ic = i0 + 4 * kg + j;
        if (ic < n) cs[(size_t)(g * G + col) * a.cap + ic] = acc[j] + 0.0f;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// k_select: exact top-k of a list's candidates
// ---------------------------------------------------------------------------
// `sel` holds the kk selected composite keys in any order.  Adds them into the
// stream's per-frame votes and fixed-point mass (scale 2^sexp, integer sums, so
// the totals do not depend on the order of the additions).  Streams of up to
// kVoteLds frames first gather the list's counts in LDS (`lv`/`lm`), so each
// (list, frame) pair costs one global atomic.  Writes the debug copy in rank
// order.
__device__ void finish_list(const ListArgs& a, int list, uint64_t* sel, int kk,
                            int32_t* lv, long long* lm) {
  const int s = list / a.NL;
  const int F = a.f[s];
  const int xs = list_mass_exponent();
  int32_t* vg = a.votes_g + (size_t)s * a.f_max;
  unsigned long long* mg = reinterpret_cast<unsigned long long*>(a.massfx_g + (size_t)s * a.f_max);
  if (F <= kVoteLds) {
    for (int f = threadIdx.x; f < F; f += blockDim.x) { lv[f] = 0; lm[f] = 0; }
    __syncthreads();
    for (int e = threadIdx.x; e < kk; e += blockDim.x) {
      const uint64_t k = sel[e];
      const int f = frame_of_row(a, s, key_row(k));
      atomicAdd(&lv[f], 1);
      atomicAdd(reinterpret_cast<unsigned long long*>(&lm[f]),
                (unsigned long long)llrint(ldexp((double)key_score(k), xs)));
    }
    __syncthreads();
    for (int f = threadIdx.x; f < F; f += blockDim.x) {
      if (lv[f] > 0) {
        atomicAdd(&vg[f], lv[f]);
        atomicAdd(&mg[f], (unsigned long long)lm[f]);
      }
    }
  } else {
    for (int e = threadIdx.x; e < kk; e += blockDim.x) {
      const uint64_t k = sel[e];
      const int f = frame_of_row(a, s, key_row(k));
      atomicAdd(&vg[f], 1);
      atomicAdd(&mg[f], (unsigned long long)llrint(ldexp((double)key_score(k), xs)));
    }
  }
  if (a.dbg_pos) {
    int32_t* dp = a.dbg_pos + (size_t)list * a.top_k;
    float* ds = a.dbg_score + (size_t)list * a.top_k;
    for (int e = threadIdx.x; e < kk; e += blockDim.x) {
      const uint64_t k = sel[e];
      int rank = 0;
      for (int e2 = 0; e2 < kk; ++e2) rank += sel[e2] > k;  // composite keys: rank order
      dp[rank] = (int32_t)key_row(k);
      ds[rank] = key_score(k);
    }
    for (int i = kk + threadIdx.x; i < a.top_k; i += blockDim.x) {
      dp[i] = -1;
      ds[i] = 0.f;
    }
  }
}

// Exact fallback for a list whose candidate count left [k, capacity]: the
// block selects from every value of the list, recomputed in each of its passes
// with the streaming pass's arithmetic (the same bits), so nothing is stored
// per row.  A pass fills `chunk` with the values of 1,024 rows (four tiles per
// wave).  Three radix rounds of 11, 11 and 10 bits over the ordered values find
// the k-th largest value v* (a round whose bin is taken whole ends the search
// early: every row at or above that bin is selected); a last pass takes the
// rows above v* and, in row order, the rows equal to it that are still needed.
constexpr int kFbTilesPerWave = 4;
constexpr int kFbRows = 16 * kFbTilesPerWave * kTile;   // rows per pass of a 1024-thread block

template <class Chunk>
__device__ void fallback_select_rows(int n, int kk, Chunk score_chunk, const float* chunk, uint64_t* sel,
                                     uint32_t* hist, uint32_t* res) {
  __shared__ uint32_t ngt_sh;
  __shared__ int scan_sh[17];
  uint32_t prefix = 0, mask = 0, need = (uint32_t)kk;
  bool whole = false;
  for (int rd = 0; rd < 3 && !whole; ++rd) {
    const int shift = rd == 0 ? 21 : rd == 1 ? 10 : 0;
    const uint32_t nb = rd == 2 ? 1024u : 2048u;
    for (int i = threadIdx.x; i < 2048; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int c0 = 0; c0 < n; c0 += kFbRows) {
      score_chunk(c0);
      __syncthreads();
      const int r = c0 + (int)threadIdx.x;
      if (r < n) {
        const uint32_t u = ord_u32(chunk[threadIdx.x]);
        if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & (nb - 1)], 1u);
      }
      __syncthreads();
    }
    if (nb == 2048u) find_digit_wide<32>(hist, need, res);
    else find_digit_wide<16>(hist, need, res);
    const uint32_t b = res[0], above = res[1], inb = res[2];
    __syncthreads();
    prefix |= b << shift;
    mask |= (nb - 1) << shift;
    need -= above;
    whole = inb == need;   // the bin is taken whole: every row >= prefix is selected
  }
  const uint32_t vstar = prefix;
  const int need_eq = whole ? 0 : (int)need;
  if (threadIdx.x == 0) ngt_sh = 0;
  __syncthreads();
  int eq_taken = 0;
  for (int c0 = 0; c0 < n; c0 += kFbRows) {
    score_chunk(c0);
    __syncthreads();
    const int r = c0 + (int)threadIdx.x;
    uint32_t u = 0;
    bool gt = false, eq = false;
    if (r < n) {
      u = ord_u32(chunk[threadIdx.x]);
      gt = whole ? u >= vstar : u > vstar;
      eq = !whole && u == vstar;
    }
    if (gt) {
      const uint32_t slot = atomicAdd(&ngt_sh, 1u);
      if (slot < (uint32_t)kMaxTopK) sel[slot] = mk_key(u, (uint32_t)r);
    }
    int tot;
    // ends with a barrier, after every thread has read its chunk entry
    const int pre = block_excl_scan(eq ? 1 : 0, scan_sh, tot);
    if (eq && eq_taken + pre < need_eq) sel[kk - need_eq + eq_taken + pre] = mk_key(u, (uint32_t)r);
    eq_taken += tot;
  }
  __syncthreads();
}

// Rewrites selected composite keys from logits to attention probabilities
// exp(s - lse) (a list keeps its order).  Ends with a barrier.
__device__ void to_probabilities(uint64_t* sel, int kk, float lse) {
  __syncthreads();
  for (int e = threadIdx.x; e < kk; e += blockDim.x) {
    const uint64_t k = sel[e];
    sel[e] = mk_key(ord_u32(__expf(key_score(k) - lse) + 0.0f), key_row(k));
  }
  __syncthreads();
}

__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <int D>
__device__ void fallback_list(const ListArgs& a, int list, uint64_t* sel, int32_t* lv, long long* lm,
                              uint32_t* res) {
  constexpr int KS = D / 32;
  __shared__ float chunk[kFbRows];
  __shared__ uint32_t max_sh;
  __shared__ unsigned long long sum_sh;
  const int s = list / a.NL, ll = list - s * a.NL;
  const int kk = a.kk[s], n = a.n[s];
  int l, g0, ng, col;
  if (a.head_mode == 0) {
    l = ll / a.Hq;
    const int h = ll - l * a.Hq;
    g0 = h / a.G;
    col = h - g0 * a.G;
    ng = 1;
  } else {
    l = ll;
    g0 = 0;
    col = 0;
    ng = a.Hk;
  }
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const int kg = lane >> 4, rl = lane & 15;
  const size_t gstride = (size_t)a.stride[s] * D;
  u32x4 bh[KS], bl[KS];
  if (a.head_mode == 0) {
    const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * a.Hk + g0) * (2 * KS * kWave);
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      bh[i] = qb[i * kWave + lane];
      bl[i] = qb[(KS + i) * kWave + lane];
    }
  } else {
    hm_load_b<KS>(a.qB + (size_t)(s * a.L + l) * a.Hk * (2 * KS * kWave), a.Hk, bh);
  }
  // chunk[r - c0] = score of row r for rows [c0, c0 + kFbRows) below n
  auto score_chunk = [&](int c0) {
#pragma unroll 1
    for (int q = 0; q < kFbTilesPerWave; ++q) {
      const int tl = wave * kFbTilesPerWave + q;        // tile of the chunk
      const int row = c0 + tl * kTile + rl;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int g = g0; g < g0 + ng; ++g) {
        const uint16_t* p = a.keys[s] + ((size_t)l * a.Hk + g) * gstride + (size_t)(row < n ? row : 0) * D + 8 * kg;
        u32x4 A[KS];
#pragma unroll
        for (int i = 0; i < KS; ++i) A[i] = row < n ? ld_nt(p + 32 * i) : u32x4{0, 0, 0, 0};
        if (a.head_mode == 0) acc = score_hilo<KS>(A, bh, bl);
        else hm_accumulate<KS>(A, bh, g, acc);   // acc gathers the per-head results
      }
      if (a.head_mode == 1) acc = hm_finish(acc);
      if ((lane & 15) == col) {
#pragma unroll
        for (int j = 0; j < 4; ++j) chunk[tl * kTile + 4 * kg + j] = acc[j] + 0.0f;
      }
    }
  };
  uint32_t* hist = reinterpret_cast<uint32_t*>(lv);   // 2048 bins; lv is free until finish_list
  fallback_select_rows(n, kk, score_chunk, chunk, sel, hist, res);
  if (a.score_mode == 1) {
    // head mode 0, attention probabilities: the list's exact log-sum-exp over
    // all its rows (the maximum, then the exp sum in fixed point), then the
    // selected rows' probabilities
    if (threadIdx.x == 0) { max_sh = 0; sum_sh = 0; }
    __syncthreads();
    uint32_t mx = 0;
    for (int c0 = 0; c0 < n; c0 += kFbRows) {
      score_chunk(c0);
      __syncthreads();
      if (c0 + (int)threadIdx.x < n) mx = max(mx, ord_u32(chunk[threadIdx.x]));
      __syncthreads();
    }
    atomicMax(&max_sh, mx);
    __syncthreads();
    const float M = ord_f32(max_sh);
    double sm = 0.0;
    for (int c0 = 0; c0 < n; c0 += kFbRows) {
      score_chunk(c0);
      __syncthreads();
      if (c0 + (int)threadIdx.x < n) sm += (double)__expf(chunk[threadIdx.x] - M);
      __syncthreads();
    }
    atomicAdd(&sum_sh, (unsigned long long)llrint(ldexp(sm, kBelowExp)));
    __syncthreads();
    to_probabilities(sel, kk, M + (float)log(ldexp((double)sum_sh, -kBelowExp)));
  }
  finish_list(a, list, sel, kk, lv, lm);
}

// Head mode 0, attention probabilities: the log-sum-exp of a list over all its
// candidate rows.  The candidates (every row at or above the cut-off tau) are
// summed here in fixed point against M = max(tau, their largest logit); the
// streaming pass summed exp(s - tau) over the rows below tau.
__device__ float lse_from_candidates(const ListArgs& a, int list, const uint64_t* src, int n, uint32_t* mm) {
  __shared__ unsigned long long fx_sh;
  const float tau = ord_f32(a.tau[list]);
  uint32_t mn = 0xFFFFFFFFu, mx = ord_u32(tau + 0.0f);
  for (int i = threadIdx.x; i < n; i += blockDim.x) mx = max(mx, (uint32_t)(src[i] >> 32));
  block_minmax_u32(mn, mx, mm);
  const float M = ord_f32(mx);
  if (threadIdx.x == 0) fx_sh = 0;
  __syncthreads();
  unsigned long long part = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x)
    part += (unsigned long long)llrint(ldexp((double)__expf(key_score(src[i]) - M), kBelowExp));
  if (part) atomicAdd(&fx_sh, part);
  __syncthreads();
  const double z = ldexp((double)fx_sh, -kBelowExp) +
                   ldexp((double)a.below[list], -kBelowExp) * exp((double)tau - (double)M);
  return M + (float)log(z);
}

// Head mode 1, attention probabilities: each head's exact log-sum-exp lse_h
// over the list, one wave per (list, head), from the candidates' logits in
// cand_sc summed in fixed point against M_h = max(Lhat_h, their largest logit)
// (so the order of the additions does not matter), plus the streaming pass's
// sum over the rows it left out (each of those added exp(s - Lhat_h) /
// (H_q tau_hat)).  Lists that take the exact fallback are skipped.
__global__ __launch_bounds__(256) void k_cand_lse(ListArgs a) {
  constexpr int kIt = 8;   // loads in flight per thread
  __shared__ float redf[4];
  __shared__ unsigned long long redu[4];
  const int list = blockIdx.x / a.Hq, h = blockIdx.x - list * a.Hq;
  const int s = list / a.NL, l = list - s * a.NL;
  const uint32_t c = a.cnt[list];
  if (c < (uint32_t)a.kk[s] || c > (uint32_t)a.cap) return;
  const int n = (int)c;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const float* ch = a.cand_sc + ((size_t)list * a.Hq + h) * a.cap;
  const size_t hb = (size_t)s * a.NLs + (size_t)l * a.Hq + h;
  const float Lh = a.lhat[hb];
  float mx = -INFINITY;
  for (int b = 0; b < n; b += 256 * kIt) {
    float x[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int i = b + it * 256 + (int)threadIdx.x;
      x[it] = i < n ? ch[i] : -INFINITY;
    }
#pragma unroll
    for (int it = 0; it < kIt; ++it) mx = fmaxf(mx, x[it]);
  }
  mx = wave_max_f32(mx);
  if (lane == 0) redf[wave] = mx;
  __syncthreads();
  const float M = fmaxf(fmaxf(fmaxf(redf[0], redf[1]), fmaxf(redf[2], redf[3])), Lh);
  unsigned long long fx = 0;
  for (int b = 0; b < n; b += 256 * kIt) {
    float x[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int i = b + it * 256 + (int)threadIdx.x;
      x[it] = i < n ? ch[i] : -INFINITY;
    }
#pragma unroll
    for (int it = 0; it < kIt; ++it)
      if (b + it * 256 + (int)threadIdx.x < n) fx += (unsigned long long)llrint(ldexp((double)__expf(x[it] - M), kBelowExp));
  }
  fx = wave_sum_u64(fx);
  if (lane == 0) redu[wave] = fx;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned long long tot = redu[0] + redu[1] + redu[2] + redu[3];
    const double tau = (double)ord_f32(a.tau[list]);
    const double left_out = ldexp((double)a.below[hb], -kBelowExp) * (double)a.Hq * tau;
    const double z = ldexp((double)tot, -kBelowExp) + left_out * exp((double)Lh - (double)M);
    a.cand_lse[(size_t)list * a.Hq + h] = M + (float)log(z);
  }
}

// Head mode 1, attention probabilities: each candidate's exact alpha =
// mean_h exp(s_h - lse_h), written into its composite key.  Returns rho =
// max_h exp(Lhat_h - lse_h): a left-out row's alpha is at most rho times its
// estimate.  Ends with a barrier.
__device__ __forceinline__ float hp_candidate_values(const ListArgs& a, int list, int n) {
  __shared__ float lse_sh[kMaxHeadsHp];
  __shared__ uint32_t rho_sh;
  const int s = list / a.NL, l = list - s * a.NL;
  const int Hq = a.Hq;
  uint64_t* src = a.cand + (size_t)list * a.cap;
  const float* cs = a.cand_sc + (size_t)list * Hq * a.cap;
  const size_t hb = (size_t)s * a.NLs + (size_t)l * Hq;
  if (threadIdx.x == 0) rho_sh = 0;
  __syncthreads();
  for (int h = threadIdx.x; h < Hq; h += blockDim.x) {
    const float lse = a.cand_lse[(size_t)list * Hq + h];
    lse_sh[h] = lse;
    atomicMax(&rho_sh, ord_u32(expf(a.lhat[hb + h] - lse)));   // positive values: the order of the floats
  }
  __syncthreads();
  const float inv_h = 1.0f / (float)Hq;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    float al = 0.f;
#pragma unroll 8
    for (int h = 0; h < Hq; ++h) al += __expf(cs[(size_t)h * a.cap + i] - lse_sh[h]);
    src[i] = mk_key(ord_u32(al * inv_h + 0.0f), key_row(src[i]));
  }
  __threadfence_block();
  __syncthreads();
  return ord_f32(rho_sh);
}

// The head-mode-1 probability selection is exact when its k-th largest value
// exceeds rho times the largest estimate alpha_hat among the rows the streaming
// pass left out (with 1e-4 of margin for the fp32 error of alpha and of its
// estimate): such a row's exact alpha is at most rho alpha_hat.  Trivially so
// when no row was left out.
__device__ bool hp_selection_proven(const ListArgs& a, int list, const uint64_t* sel, int kk, float rho,
                                    uint32_t* mm) {
  uint32_t mn = 0xFFFFFFFFu, mx = 0;
  for (int e = threadIdx.x; e < kk; e += blockDim.x) mn = min(mn, (uint32_t)(sel[e] >> 32));
  block_minmax_u32(mn, mx, mm);
  const uint32_t lm = a.left_max[list];
  if (lm == 0) return true;
  return ord_f32(mn) > ord_f32(lm) * rho * 1.0001f;
}

// Head mode 1 with attention probabilities, exact over every row of the list
// (when the candidate count left [k, capacity] or the selection could not be
// proven).  Pass 1 takes each head's largest logit, pass 2 its exp sum against
// it (fixed point, so the order of the additions does not matter): the exact
// lse_h.  The rows are then selected by alpha = mean_h exp(s_h - lse_h) with
// the radix rounds above, every pass recomputing the logits with the streaming
// pass's arithmetic.
template <int D>
__device__ void fallback_list_hp(const ListArgs& a, int list, uint64_t* sel, int32_t* lv, long long* lm,
                                 uint32_t* res) {
  constexpr int KS = D / 32;
  __shared__ float chunk[kFbRows];
  __shared__ uint32_t hmax[kMaxHeadsHp];
  __shared__ unsigned long long hsum[kMaxHeadsHp];
  __shared__ float lse_sh[kMaxHeadsHp];
  const int s = list / a.NL, l = list - s * a.NL;
  const int kk = a.kk[s], n = a.n[s], Hq = a.Hq, G = a.G, Hk = a.Hk;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
  const int kg = lane >> 4, rl = lane & 15, col = lane & 15;
  const size_t gstride = (size_t)a.stride[s] * D;
  // logits of KV head g for tile t: lane (c, kg) gets head g G + c, rows 16 t + 4 kg + j
  auto tile_logits = [&](int t, int g) -> f32x4 {
    const int row = t * kTile + rl;
    const u32x4* qb = a.qB + ((size_t)(s * a.L + l) * Hk + g) * (2 * KS * kWave);
    const uint16_t* p = a.keys[s] + ((size_t)l * Hk + g) * gstride + (size_t)(row < n ? row : 0) * D + 8 * kg;
    u32x4 bh[KS], bl[KS], A[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
      bh[i] = qb[i * kWave + lane];
      bl[i] = qb[(KS + i) * kWave + lane];
      A[i] = row < n ? ld_nt(p + 32 * i) : u32x4{0, 0, 0, 0};
    }
    return score_hilo<KS>(A, bh, bl);
  };
  for (int h = threadIdx.x; h < Hq; h += blockDim.x) { hmax[h] = 0; hsum[h] = 0; }
  __syncthreads();
  // pass 1: every head's largest logit (one KV head at a time, which keeps
  // the registers of one head's running values)
  const int ntile = (n + kTile - 1) / kTile;
#pragma unroll 1
  for (int g = 0; g < Hk; ++g) {
    float mx = -INFINITY;
    for (int t = wave; t < ntile; t += blockDim.x / kWave) {
      const f32x4 acc = tile_logits(t, g);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (t * kTile + 4 * kg + j < n) mx = fmaxf(mx, acc[j]);
    }
    if (col < G && mx > -INFINITY) atomicMax(&hmax[g * G + col], ord_u32(mx));
  }
  __syncthreads();
  // pass 2: every head's exp sum against its maximum (a wave's sum over its
  // tiles in fp64, then added in fixed point)
#pragma unroll 1
  for (int g = 0; g < Hk; ++g) {
    double sm = 0.0;
    const float M = col < G ? ord_f32(hmax[g * G + col]) : 0.f;
    for (int t = wave; t < ntile; t += blockDim.x / kWave) {
      const f32x4 acc = tile_logits(t, g);   // uniform: the whole wave issues the loads and MFMAs
      if (col < G) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (t * kTile + 4 * kg + j < n) sm += (double)__expf(acc[j] - M);
      }
    }
    if (col < G && sm > 0.0) atomicAdd(&hsum[g * G + col], (unsigned long long)llrint(ldexp(sm, kBelowExp)));
  }
  __syncthreads();
  for (int h = threadIdx.x; h < Hq; h += blockDim.x)
    lse_sh[h] = ord_f32(hmax[h]) + (float)log(ldexp((double)hsum[h], -kBelowExp));
  __syncthreads();
  const float inv_h = 1.0f / (float)Hq;
  // chunk[r - c0] = alpha of row r for rows [c0, c0 + kFbRows) below n
  auto alpha_chunk = [&](int c0) {
#pragma unroll
    for (int q = 0; q < kFbTilesPerWave; ++q) {
      const int tl = wave * kFbTilesPerWave + q;
      const int t = c0 / kTile + tl;
      f32x4 rs = {0.f, 0.f, 0.f, 0.f};
      for (int g = 0; g < Hk; ++g) {
        const f32x4 acc = tile_logits(t, g);
        const float L = col < G ? lse_sh[g * G + col] : INFINITY;
#pragma unroll
        for (int j = 0; j < 4; ++j) rs[j] += __expf(acc[j] - L);
      }
      rs = hm_finish(rs);
      if (col == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) chunk[tl * kTile + 4 * kg + j] = rs[j] * inv_h + 0.0f;
      }
    }
  };
  uint32_t* hist = reinterpret_cast<uint32_t*>(lv);
  fallback_select_rows(n, kk, alpha_chunk, chunk, sel, hist, res);
  finish_list(a, list, sel, kk, lv, lm);
}

// LDS of one list's selection.
struct SelectShared {
  uint64_t sel[kMaxTopK];
  int32_t lv[kVoteLds];
  long long lm[kVoteLds];
};

// The register path of select_candidates: N candidates per thread (of 1024);
// the values (high halves) and inverted rows in registers: the k-th value,
// then the cut among the ties at that value by row.
// Exact top-kk of the n keys the block holds in registers (key it of thread t
// is candidate t + 1024 it; keys past n are ignored) into `sel`.
template <int N>
__device__ __forceinline__ void select_from_keys(const uint64_t (&key)[N], int n, int kk, uint64_t* sel,
                                                 uint32_t* hist, uint32_t* res, uint32_t& ngather,
                                                 uint32_t* mm) {
  uint32_t u[N], w[N];
  bool ok[N], tie[N];
  uint32_t mn = 0xFFFFFFFFu, mx = 0;
#pragma unroll
  for (int it = 0; it < N; ++it) {
    const int i = threadIdx.x + it * 1024;
    ok[it] = i < n;
    const uint64_t k = ok[it] ? key[it] : 0;
    u[it] = (uint32_t)(k >> 32);
    w[it] = (uint32_t)k;  // 0xFFFFFFFF - row: larger for lower rows
    if (ok[it]) { mn = min(mn, u[it]); mx = max(mx, u[it]); }
  }
  block_minmax_u32(mn, mx, mm);
  uint32_t n_gt, n_eq;
  const uint32_t vstar = block_select_range<N, false>(u, ok, mn, mx, (uint32_t)kk, hist, res, n_gt, n_eq);
  const uint32_t need = (uint32_t)kk - n_gt;
  uint32_t wcut = 0;  // ties with w >= wcut (the `need` lowest rows) are taken
  if (n_eq > need) {
    uint32_t wmin = 0xFFFFFFFFu, wmax = 0;
#pragma unroll
    for (int it = 0; it < N; ++it) {
      tie[it] = ok[it] && u[it] == vstar;
      if (tie[it]) { wmin = min(wmin, w[it]); wmax = max(wmax, w[it]); }
    }
    block_minmax_u32(wmin, wmax, mm);
    uint32_t g2, e2;
    wcut = block_select_range<N, false>(w, tie, wmin, wmax, need, hist, res, g2, e2);
  }
#pragma unroll
  for (int it = 0; it < N; ++it) {
    if (ok[it] && (u[it] > vstar || (u[it] == vstar && w[it] >= wcut))) {
      const uint32_t slot = atomicAdd(&ngather, 1u);
      if (slot < (uint32_t)kMaxTopK) sel[slot] = ((uint64_t)u[it] << 32) | w[it];
    }
  }
}

template <int N>
__device__ __forceinline__ void select_in_registers(const uint64_t* src, int n, int kk, uint64_t* sel,
                                                    uint32_t* hist, uint32_t* res, uint32_t& ngather,
                                                    uint32_t* mm) {
  uint64_t key[N];
#pragma unroll
  for (int it = 0; it < N; ++it) {
    const int i = threadIdx.x + it * 1024;
    key[it] = i < n ? src[i] : 0;
  }
  select_from_keys<N>(key, n, kk, sel, hist, res, ngather, mm);
}

// Exact top-kk of a list's n candidate keys (composite: value, then row) into
// `sel`, in any order: in registers for up to 8,192 candidates (4 per thread up
// to 4,096, so that the passes over them issue no idle slots), else a radix
// selection over the keys in global memory.  Ends with a barrier.
__device__ __forceinline__ void select_candidates(const uint64_t* src, int n, int kk, uint64_t* sel, uint32_t* hist,
                                                  uint32_t* res, uint32_t& ngather, uint32_t* mm) {
  if (threadIdx.x == 0) ngather = 0;
  if (n <= 1024 * 4) {
    select_in_registers<4>(src, n, kk, sel, hist, res, ngather, mm);
  } else if (n <= 1024 * kSelItems) {
    select_in_registers<kSelItems>(src, n, kk, sel, hist, res, ngather, mm);
  } else {
    // large candidate sets: radix select over the keys in global memory
    __syncthreads();
    const uint64_t cut = radix_select_u64([&](int i) { return src[i]; }, n, (uint32_t)kk, hist, res);
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      const uint64_t x = src[i];
      if (x >= cut) {
        const uint32_t slot = atomicAdd(&ngather, 1u);
        if (slot < (uint32_t)kMaxTopK) sel[slot] = x;
      }
    }
  }
  __syncthreads();
}

// HP: head mode 1 with attention probabilities (its own kernel, so that the
// registers and LDS of its paths stay out of the other modes' selection).
template <int D, bool HP>
__device__ void select_list(const ListArgs& a, int list, SelectShared& sh, uint32_t* hist, uint32_t* res,
                            uint32_t& ngather, uint32_t* mm) {
  uint64_t* sel = sh.sel;
  int32_t* lv = sh.lv;
  long long* lm = sh.lm;
  const int s = list / a.NL;
  const int kk = a.kk[s];
  if (kk == 0) {   // no rows: nothing is voted, the exponent only has to be finite
    if (threadIdx.x == 0 && list == s * a.NL) a.sexp[s] = 0;
    finish_list(a, list, sel, 0, lv, lm);
    return;
  }
  const uint32_t c = a.cnt[list];
  uint64_t* src = a.cand + (size_t)list * a.cap;
  // the first 4,096 candidate slots are read together with the count (from
  // clamped in-bounds slots; slots past the count are ignored): one round trip
  // instead of two for the usual list
  uint64_t pre[4];
  if (!HP) {
#pragma unroll
    for (int it = 0; it < 4; ++it) pre[it] = src[min((int)threadIdx.x + it * 1024, a.cap - 1)];
  }
  // the stream's mass exponent, by wave 0 while the candidates load (every
  // path below passes block barriers before finish_list reads it); the
  // stream's first list publishes it for the pool
  if (threadIdx.x < kWave) {
    const int xs = stream_exponent(a, s);
    if (threadIdx.x == 0) {
      list_mass_exponent() = xs;
      if (list == s * a.NL) a.sexp[s] = xs;
    }
  }
  int fallback = (c < (uint32_t)kk || c > (uint32_t)a.cap) ? 1 : 0;
  float rho = 0.f;
  if (HP && !fallback) rho = hp_candidate_values(a, list, (int)c);
  if (!fallback) {
    if (!HP && c <= 4096u) {
      if (threadIdx.x == 0) ngather = 0;
      select_from_keys<4>(pre, (int)c, kk, sel, hist, res, ngather, mm);
      __syncthreads();
    } else {
      select_candidates(src, (int)c, kk, sel, hist, res, ngather, mm);
    }
    // head mode 1, attention probabilities: the selection is exact when its
    // k-th value beats every row the streaming pass left out (fallback 2)
    if (HP && !hp_selection_proven(a, list, sel, kk, rho, mm)) fallback = 2;
  }
  if (a.dbg_stats && threadIdx.x == 0) {
    a.dbg_stats[2 * list] = (int32_t)min(c, (uint32_t)INT_MAX);
    a.dbg_stats[2 * list + 1] = fallback;
  }
  if (fallback) {
    if (HP) fallback_list_hp<D>(a, list, sel, lv, lm, res);
    else fallback_list<D>(a, list, sel, lv, lm, res);
    return;
  }
  if (!HP && a.score_mode == 1) {
    // head mode 0: the lists are those of the logits; the normaliser of the
    // list is the candidates' exp sum plus the streaming pass's sum below the
    // cut-off, and the selected rows carry their probabilities from here on
    const float lse = lse_from_candidates(a, list, src, (int)c, mm);
    to_probabilities(sel, kk, lse);
  }
  finish_list(a, list, sel, kk, lv, lm);
}

// ---------------------------------------------------------------------------
// k_votes_pool: votes, attention mass and the vote-ranked pool (one block per stream)
// ---------------------------------------------------------------------------
struct VoteArgs {
  int NL, k_max, pool, f_max, hist_stride;
  int32_t f[kMaxStreams];
  int64_t frame0[kMaxStreams];   // id of the first candidate frame (pool ids are reported as absolute ids)
  int64_t hist0[kMaxStreams];    // its place among the stored frames (index of the debug histograms)
  const int32_t* votes_g;    // [S][f_max] per-frame votes
  const int64_t* massfx_g;   // [S][f_max] per-frame mass at scale 2^sexp[s]
  const int32_t* sexp;       // [S]
  uint64_t* rec_hi;     // [S][f_max] compacted records
  uint64_t* rec_lo;
  int32_t* pool_ids;    // [S][pool]
  int32_t* pool_votes;  // [S][pool]
  float* pool_mass;     // [S][pool]
  int32_t* pool_n;
  int32_t* dbg_vote_hist;
  float* dbg_mass_hist;
  int32_t* dbg_pool;
  int32_t* dbg_pool_n;
};

// The pool: the voted frames of rank < pool by (votes desc, mass desc, frame
// asc) from the per-frame votes and fixed-point masses that the selection
// blocks accumulated, ranked by counting.
//
// Records: hi = votes:32 | mass_hi:32, lo = mass_lo:32 | ~frame:32, compared
// descending (mass as offset binary).  The cut between the pool and the rest:
// a histogram of the votes gives the vote count v* of the last pool slot; the
// frames with exactly v* votes are ranked by counting among themselves (when
// there are at most kTieRank of them, the usual case); otherwise a radix cut
// over the 128-bit records.  Leaves the ordered pool in shi/slo[0 .. pn) and
// returns pn.  One block of 1024 threads per stream.
constexpr int kVoteBins = 2048;   // vote histogram bins (the last one collects larger counts)
constexpr int kTieRank = 128;     // frames tied at the cut ranked by counting

struct PoolShared {
  uint64_t shi[kPoolSort];
  uint64_t slo[kPoolSort];
  uint64_t ghi[kMaxPool];
  uint64_t glo[kMaxPool];
  uint32_t vh[kVoteBins];
  int tl[kTieRank];
  int scan[17];
  uint32_t hist[256];
  uint32_t res[4];
  uint32_t nvoted, ngather, ntie;
  uint64_t cut_hi, cut_lo;
  int vstar, above, inb;
};

// `lds_ids` (optional, kMaxPool entries) receives the ordered pool's frame ids
// for the caller's block; with `write_out` false the block writes nothing to
// global memory (several blocks of a stream may rank the same pool, and then
// only one publishes it; its records must then fit in LDS: at most kPoolSort
// candidate frames).
__device__ int pool_select(const VoteArgs& a, int s, PoolShared& sh, int* lds_ids = nullptr,
                           bool write_out = true) {
  const int F = a.f[s];
  const int32_t* votes = a.votes_g + (size_t)s * a.f_max;
  const int64_t* massfx = a.massfx_g + (size_t)s * a.f_max;
  if (threadIdx.x == 0) { sh.nvoted = 0; sh.ngather = 0; sh.ntie = 0; sh.vstar = -1; }
  __syncthreads();
  const double inv = ldexp(1.0, -a.sexp[s]);
  uint64_t* rh = a.rec_hi + (size_t)s * a.f_max;
  uint64_t* rl = a.rec_lo + (size_t)s * a.f_max;
  // four frames per thread per pass, their loads issued together; every lane of a
  // wave takes part in the ballots (frames past F count as unvoted)
  for (int f0 = 0; f0 < F; f0 += 4 * (int)blockDim.x) {
    int vv[4];
    int64_t mm[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int f = f0 + u * (int)blockDim.x + (int)threadIdx.x;
      vv[u] = f < F ? votes[f] : 0;
      mm[u] = f < F ? massfx[f] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int f = f0 + u * (int)blockDim.x + (int)threadIdx.x;
      const int v = vv[u];
      const int64_t mf = mm[u];
      if (write_out && a.dbg_vote_hist && f < F) {
        a.dbg_vote_hist[(size_t)s * a.hist_stride + a.hist0[s] + f] = v;
        a.dbg_mass_hist[(size_t)s * a.hist_stride + a.hist0[s] + f] = (float)((double)mf * inv);
      }
      // one LDS atomic per wave for the wave's voted frames
      const uint64_t vm = __ballot(v >= 1);
      if (vm == 0) continue;
      const int first = __builtin_ffsll((long long)vm) - 1;
      uint32_t base = 0;
      if ((threadIdx.x & 63) == (uint32_t)first) base = atomicAdd(&sh.nvoted, (uint32_t)__popcll(vm));
      base = __shfl(base, first);
      if (v >= 1) {
        const uint32_t slot = base + (uint32_t)__popcll(vm & ((1ull << (threadIdx.x & 63)) - 1ull));
        const uint64_t mb = (uint64_t)mf ^ 0x8000000000000000ull;
        const uint64_t h = ((uint64_t)(uint32_t)v << 32) | (mb >> 32);
        const uint64_t l = (mb << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)f);
        if (slot < (uint32_t)kPoolSort) { sh.shi[slot] = h; sh.slo[slot] = l; }
        else { rh[slot] = h; rl[slot] = l; }
      }
    }
  }
  if (write_out && a.dbg_vote_hist) {
    for (int f = threadIdx.x; f < a.hist_stride; f += blockDim.x) {
      if (f >= a.hist0[s] && f < a.hist0[s] + F) continue;
      a.dbg_vote_hist[(size_t)s * a.hist_stride + f] = 0;
      a.dbg_mass_hist[(size_t)s * a.hist_stride + f] = 0.f;
    }
  }
  __syncthreads();
  const int n_voted = (int)sh.nvoted;
  const int P = a.pool;
  const int pn = min(P, n_voted);
  const bool in_lds = n_voted <= kPoolSort;
  if (!in_lds) {   // the records beyond the LDS part live in global memory only
    for (int i = threadIdx.x; i < kPoolSort; i += blockDim.x) { rh[i] = sh.shi[i]; rl[i] = sh.slo[i]; }
    __threadfence();   // every record, from any thread, visible to the reads below
    __syncthreads();
  }
  auto get = [&](int i, uint64_t& h, uint64_t& l) {
    if (in_lds) { h = sh.shi[i]; l = sh.slo[i]; }
    else {
      h = __hip_atomic_load(&rh[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      l = __hip_atomic_load(&rl[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  };
  uint64_t ch = 0, cl = 0;
  if (n_voted > P) {
    bool cut = false;
    if (in_lds) {
      // vote histogram; pair of bins (2q, 2q + 1) per thread, q from the top
      for (int i = threadIdx.x; i < kVoteBins; i += blockDim.x) sh.vh[i] = 0;
      __syncthreads();
      for (int i = threadIdx.x; i < n_voted; i += blockDim.x)
        atomicAdd(&sh.vh[min((uint32_t)(sh.shi[i] >> 32), (uint32_t)(kVoteBins - 1))], 1u);
      __syncthreads();
      const int q = kVoteBins / 2 - 1 - (int)threadIdx.x;   // blockDim == kVoteBins / 2
      const int hb = (int)sh.vh[2 * q + 1], lb = (int)sh.vh[2 * q];
      int tot;
      const int above = block_excl_scan(hb + lb, sh.scan, tot);   // records in higher bin pairs
      if (above < P && P <= above + hb) { sh.vstar = 2 * q + 1; sh.above = above; sh.inb = hb; }
      else if (above + hb < P && P <= above + hb + lb) { sh.vstar = 2 * q; sh.above = above + hb; sh.inb = lb; }
      __syncthreads();
      const int vstar = sh.vstar, need = P - sh.above, inb = sh.inb;
      if (vstar >= 1 && vstar < kVoteBins - 1 && inb <= kTieRank) {
        if (inb == need) {
          ch = (uint64_t)(uint32_t)vstar << 32;   // every frame with >= v* votes
          cl = 0;
        } else {
          for (int i = threadIdx.x; i < n_voted; i += blockDim.x)
            if ((int)(sh.shi[i] >> 32) == vstar) sh.tl[atomicAdd(&sh.ntie, 1u)] = i;
          __syncthreads();
          if ((int)threadIdx.x < inb) {
            const int me = sh.tl[threadIdx.x];
            const uint64_t h = sh.shi[me], l = sh.slo[me];
            int rank = 0;
            for (int k = 0; k < inb; ++k) {
              const int o = sh.tl[k];
              rank += rec_less(h, l, sh.shi[o], sh.slo[o]);
            }
            if (rank == need - 1) { sh.cut_hi = h; sh.cut_lo = l; }   // records are distinct
          }
          __syncthreads();
          ch = sh.cut_hi;
          cl = sh.cut_lo;
        }
        cut = true;
      }
    }
    if (!cut) radix_select_u128(get, n_voted, (uint32_t)P, sh.hist, sh.res, ch, cl);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < n_voted; i += blockDim.x) {
    uint64_t h, l;
    get(i, h, l);
    if (h > ch || (h == ch && l >= cl)) {
      const uint32_t slot = atomicAdd(&sh.ngather, 1u);
      if (slot < (uint32_t)kMaxPool) { sh.ghi[slot] = h; sh.glo[slot] = l; }
    }
  }
  __syncthreads();
  // rank by counting, 8 threads per record (pn <= kMaxPool = 256 = blockDim / 8 * 2)
  for (int i0 = 0; i0 < pn; i0 += (int)blockDim.x / 8) {
    const int i = i0 + (int)threadIdx.x / 8, part = threadIdx.x & 7;
    int rank = 0;
    uint64_t h = 0, l = 0;
    if (i < pn) {
      h = sh.ghi[i];
      l = sh.glo[i];
      for (int j = part; j < pn; j += 8) rank += rec_less(h, l, sh.ghi[j], sh.glo[j]);
    }
    rank += __shfl_xor(rank, 1);
    rank += __shfl_xor(rank, 2);
    rank += __shfl_xor(rank, 4);
    if (i < pn && part == 0) {
      sh.shi[rank] = h;   // records are distinct: ranks form a permutation
      sh.slo[rank] = l;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    int id = -1, v = 0;
    float m = 0.f;
    if (i < pn) {
      id = (int)(0xFFFFFFFFu - (uint32_t)sh.slo[i]);
      v = (int)(sh.shi[i] >> 32);
      const uint64_t mb = (sh.shi[i] << 32) | (sh.slo[i] >> 32);
      m = (float)((double)(int64_t)(mb ^ 0x8000000000000000ull) * inv);
      if (lds_ids) lds_ids[i] = id;
    }
    if (!write_out) continue;
    a.pool_ids[(size_t)s * P + i] = id;
    a.pool_votes[(size_t)s * P + i] = v;
    a.pool_mass[(size_t)s * P + i] = m;
    if (a.dbg_pool) a.dbg_pool[(size_t)s * P + i] = id >= 0 ? (int32_t)(id + a.frame0[s]) : -1;
  }
  if (write_out && threadIdx.x == 0) {
    a.pool_n[s] = pn;
    if (a.dbg_pool_n) a.dbg_pool_n[s] = pn;
  }
  return pn;
}


// One block per list: exact top-k and the list's votes and mass.
template <int D>
__global__ __launch_bounds__(1024) void k_select(ListArgs a) {
  __shared__ SelectShared sh;
  __shared__ uint32_t hist[512];
  __shared__ uint32_t res[4];
  __shared__ uint32_t ngather;
  __shared__ uint32_t mm[32];
  select_list<D, false>(a, blockIdx.x, sh, hist, res, ngather, mm);
}
// The same at two blocks per CU (64 VGPRs), for batches with more lists than
// two per CU.
template <int D>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8, 8))) void k_select_dense(ListArgs a) {
  __shared__ SelectShared sh;
  __shared__ uint32_t hist[512];
  __shared__ uint32_t res[4];
  __shared__ uint32_t ngather;
  __shared__ uint32_t mm[32];
  select_list<D, false>(a, blockIdx.x, sh, hist, res, ngather, mm);
}

// The same for head mode 1 with attention probabilities.
template <int D>
__global__ __launch_bounds__(1024) void k_select_hp(ListArgs a) {
  __shared__ SelectShared sh;
  __shared__ uint32_t hist[512];
  __shared__ uint32_t res[4];
  __shared__ uint32_t ngather;
  __shared__ uint32_t mm[32];
  select_list<D, true>(a, blockIdx.x, sh, hist, res, ngather, mm);
}

// One block per stream: the pool.
__global__ __launch_bounds__(1024) void k_votes_pool(VoteArgs a) {
  __shared__ PoolShared sh;
  pool_select(a, blockIdx.x, sh);
}

// ---------------------------------------------------------------------------
// Max-min diversity over the pool (greedy, on the Gram matrix of the pool's
// descriptors)
// ---------------------------------------------------------------------------
struct MaxminArgs {
  int pool, ld, n_select;
  int64_t frame0[kMaxStreams];   // added to the (window-relative) pool ids on output
  const int32_t* pool_ids;
  const int32_t* pool_votes;
  const float* pool_mass;
  const int32_t* pool_n;
  const float* gram;
  int64_t* out_ids;
  int32_t* out_votes;
  float* out_mass;
  int32_t* out_n;
};

// Seeded with pool rank 0; each next pick maximises its smallest distance
// 1 - k_u.k_s to the picks so far, ties to the earlier pool rank.  Pools of up
// to 128 frames run in one wave over the distances staged in LDS as
// order-preserving words (so the running minimum and the argmax are integer
// operations on the same fp32 values).
struct MaxminShared {
  uint32_t d_lds[kGramLdsPool * kGramLdsPool];
  int32_t pid[kGramLdsPool];
  int32_t pvotes[kGramLdsPool];
  float pmass[kGramLdsPool];
  float mind[kMaxPool];
  int taken[kMaxPool];
  int sel[kMaxSelect];
  float shv[16];
  int shi[16];
};

// Wave maximum left in every lane: DPP within rows of 16 lanes, then gfx950's
// row swaps (the max of a value and its swapped partner needs no lane select),
// all on the vector unit.
__device__ __forceinline__ uint32_t wave_max_all_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false));  // row_ror 4
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false));  // row_ror 8
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = max(v, max((uint32_t)r[0], (uint32_t)r[1]));
  r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return max(v, max((uint32_t)r[0], (uint32_t)r[1]));
}

// The greedy over distance words d_lds[r * kGramLdsPool + c] = ord(1 - g_rc)
// of a pool of pn <= kGramLdsPool frames, with d_lds[r * kGramLdsPool + r] = 0
// (entries of columns >= pn are never used): the first K picks into sel.  Run
// by wave 0 of the block.  Lane l holds pool ranks l and l + 64; picked and
// absent ranks hold 0 (a pick's own row zeroes it), below every distance
// word, so min() keeps them out of every later argmax; argmax by a wave max,
// ties to the lowest rank through ballots; lane i keeps the i-th pick.
__device__ __forceinline__ void maxmin_greedy_lds(const uint32_t* d_lds, int pn, int K, int* sel) {
  if (threadIdx.x >= kWave) return;
  const int lane = threadIdx.x;
  uint32_t m0 = (lane > 0 && lane < pn) ? d_lds[lane] : 0u;
  uint32_t m1 = lane + kWave < pn ? d_lds[lane + kWave] : 0u;
  int pick = 0;
  for (int it = 1; it < K; ++it) {
    const uint32_t best = wave_max_all_u32(max(m0, m1));
    const uint64_t b0 = __ballot(m0 == best), b1 = __ballot(m1 == best);
    const int bi = b0 ? __builtin_ctzll(b0) : kWave + __builtin_ctzll(b1);
    const uint32_t* row = d_lds + bi * kGramLdsPool;
    m0 = min(m0, row[lane]);
    m1 = min(m1, row[lane + kWave]);
    pick = lane == it ? bi : pick;
  }
  if (lane < K) sel[lane] = pick;
}

// The K picks in selection order (pool ranks in sel), -1 padded to n_select;
// ids, votes and mass of the stream's pool by rank.
__device__ __forceinline__ void maxmin_write(const MaxminArgs& a, int s, int K, const int* sel, const int32_t* ids,
                                             const int32_t* votes, const float* mass) {
  for (int i = threadIdx.x; i < a.n_select; i += blockDim.x) {
    const size_t o = (size_t)s * a.n_select + i;
    if (i < K) {
      const int p = sel[i];
      a.out_ids[o] = ids[p] + a.frame0[s];
      a.out_votes[o] = votes[p];
      a.out_mass[o] = mass[p];
    } else {
      a.out_ids[o] = -1;
      a.out_votes[o] = 0;
      a.out_mass[o] = 0.f;
    }
  }
  if (threadIdx.x == 0) a.out_n[s] = K;
}

__device__ void maxmin_block(const MaxminArgs& a, int s, MaxminShared& sh) {
  uint32_t* d_lds = sh.d_lds;
  float* mind = sh.mind;
  int* taken = sh.taken;
  int* sel = sh.sel;
  float* shv = sh.shv;
  int* shi = sh.shi;
  const float* G = a.gram + (size_t)s * a.pool * a.ld;
  if (a.pool <= kGramLdsPool) {
    // row r, column c < 128: ord(1 - g_rc) for c < pn, c != r, else 0 (below
    // every distance word, like a frame already picked).  Every row of the
    // pool's capacity is read at once, with the pool size, as float4 from
    // clamped in-bounds addresses (ld % 4 == 0, ld >= pool); what a clamped
    // read or a row past the pool returns is never used.
    constexpr int C4 = kGramLdsPool / 4;
    const int nq = a.pool * C4;   // <= 4 float4 per thread
    const int pn = a.pool_n[s];
    const int t = threadIdx.x;    // the pool by rank, loaded with the matrix
    int32_t pid = 0, pv = 0;
    float pm = 0.f;
    if (t < a.pool) {
      pid = a.pool_ids[(size_t)s * a.pool + t];
      pv = a.pool_votes[(size_t)s * a.pool + t];
      pm = a.pool_mass[(size_t)s * a.pool + t];
    }
    float4 x[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = min(u * (int)blockDim.x + (int)threadIdx.x, nq - 1);
      const int r = i / C4, c = min(4 * (i - r * C4), a.ld - 4);
      x[u] = *reinterpret_cast<const float4*>(G + (size_t)r * a.ld + c);
    }
    const int K = min(a.n_select, pn);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = u * blockDim.x + threadIdx.x;
      if (i < nq) {
        const int r = i / C4, c = 4 * (i - r * C4);
        const float xv[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
        uint4 o;
        uint32_t* ov = reinterpret_cast<uint32_t*>(&o);
#pragma unroll
        for (int q = 0; q < 4; ++q) ov[q] = (c + q < pn && c + q != r) ? ord_u32(1.0f - xv[q]) : 0u;
        *reinterpret_cast<uint4*>(d_lds + r * kGramLdsPool + c) = o;
      }
    }
    if (t < a.pool) { sh.pid[t] = pid; sh.pvotes[t] = pv; sh.pmass[t] = pm; }
    __syncthreads();
    maxmin_greedy_lds(d_lds, pn, K, sel);
    __syncthreads();
    maxmin_write(a, s, K, sel, sh.pid, sh.pvotes, sh.pmass);
    return;
  }
  const int pn = a.pool_n[s];
  const int K = min(a.n_select, pn);
  {
    for (int u = threadIdx.x; u < pn; u += blockDim.x) {
      mind[u] = 1.0f - G[u];          // distance to pool rank 0
      taken[u] = (u == 0);
    }
    if (threadIdx.x == 0 && K > 0) sel[0] = 0;
    __syncthreads();
    for (int it = 1; it < K; ++it) {
      float bv = -INFINITY;
      int bi = INT_MAX;
      for (int u = threadIdx.x; u < pn; u += blockDim.x) {
        if (!taken[u] && (mind[u] > bv || (mind[u] == bv && u < bi))) { bv = mind[u]; bi = u; }
      }
      const int w = block_argmax(bv, bi, shv, shi);
      for (int u = threadIdx.x; u < pn; u += blockDim.x) {
        mind[u] = fminf(mind[u], 1.0f - G[(size_t)w * a.ld + u]);
        if (u == w) taken[u] = 1;
      }
      if (threadIdx.x == 0) sel[it] = w;
      __syncthreads();
    }
  }
  maxmin_write(a, s, K, sel, a.pool_ids + (size_t)s * a.pool, a.pool_votes + (size_t)s * a.pool,
               a.pool_mass + (size_t)s * a.pool);
}

__global__ __launch_bounds__(1024) void k_maxmin(MaxminArgs a) {
  __shared__ MaxminShared sh;
  maxmin_block(a, blockIdx.x, sh);
}

// ---------------------------------------------------------------------------
// k_gram: fp32 Gram matrix of the pool descriptors, one 16 x 16 tile of the
// upper triangle per block (mirrored on store), on the fp32 MFMA 16x16x4.  Lane l
// feeds row l & 15 of either operand with dimensions 4 (l >> 4) + j of each
// 16-dimension step (j = 0..3, one MFMA each); each of the four waves covers a
// quarter of the dimensions and the four partial tiles are added in wave order.
// ---------------------------------------------------------------------------
struct GramArgs {
  int pool, ld, dim, tiles;   // ld: Gram row stride, a multiple of 4; dim in {64, 128, ..., 1024}
  const float* desc[kMaxStreams];
  const int32_t* pool_ids;
  const int32_t* pool_n;
  float* gram;          // [S][pool][ld]
};

// Tile (ti, tj) of stream s from the pool's frame ids `ids` (pn of them);
// called by the whole block, waves 0..3 compute, `part` is 4 KiB of LDS.
template <int NST>   // 16-dimension steps per wave: dim / 64
__device__ __forceinline__ void gram_tile(const GramArgs& a, int s, int ti, int tj, int pn,
                                          const int32_t* ids, float (*part)[256]) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  constexpr int dim = 64 * NST;
  if (w < 4) {
    // rows past the pool repeat its last row: they only feed tile entries that
    // are never stored
    const int ri = min(ti * 16 + (lane & 15), pn - 1), rj = min(tj * 16 + (lane & 15), pn - 1);
    const float* xi = a.desc[s] + (size_t)ids[ri] * dim + w * (dim / 4) + 4 * (lane >> 4);
    const float* xj = a.desc[s] + (size_t)ids[rj] * dim + w * (dim / 4) + 4 * (lane >> 4);
    float4 va[NST], vb[NST];
#pragma unroll
    for (int u = 0; u < NST; ++u) {
      va[u] = *reinterpret_cast<const float4*>(xi + 16 * u);
      vb[u] = *reinterpret_cast<const float4*>(xj + 16 * u);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < NST; ++u) {
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(va[u].x, vb[u].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(va[u].y, vb[u].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(va[u].z, vb[u].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(va[u].w, vb[u].w, acc, 0, 0, 0);
    }
    // lane l holds tile rows 4 (l >> 4) + j, column l & 15
#pragma unroll
    for (int j = 0; j < 4; ++j) part[w][(4 * (lane >> 4) + j) * 16 + (lane & 15)] = acc[j];
  }
  __syncthreads();
  if (threadIdx.x < 256) {
    const int r = threadIdx.x >> 4, c = threadIdx.x & 15;
    const float v = ((part[0][threadIdx.x] + part[1][threadIdx.x]) + part[2][threadIdx.x]) + part[3][threadIdx.x];
    const int pi = ti * 16 + r, pj = tj * 16 + c;
    if (pi < pn && pj < pn) {
      float* G = a.gram + (size_t)s * a.pool * a.ld;
      G[(size_t)pi * a.ld + pj] = v;
      G[(size_t)pj * a.ld + pi] = v;
    }
  }
}

template <int NST>
__global__ __launch_bounds__(256) void k_gram(GramArgs a) {
  __shared__ float part[4][256];
  const int s = blockIdx.x / (a.tiles * a.tiles);
  const int t = blockIdx.x % (a.tiles * a.tiles);
  const int ti = t / a.tiles, tj = t % a.tiles;
  const int pn = a.pool_n[s];
  if (tj < ti || ti * 16 >= pn || tj * 16 >= pn) return;
  gram_tile<NST>(a, s, ti, tj, pn, a.pool_ids + (size_t)s * a.pool, part);
}

// The pool and its Gram matrix in one launch, for streams of at most kPoolSort
// candidate frames: every block of the upper triangle ranks the stream's pool
// itself (the same records, so the same pool) and computes its tile from the
// ids in LDS; tile (0, 0) publishes the pool.  This saves the pool kernel's
// launch and the Gram blocks' read of the pool ids.
template <int NST>
__global__ __launch_bounds__(1024) void k_pool_gram(VoteArgs va, GramArgs a) {
  __shared__ PoolShared psh;
  __shared__ int32_t ids[kMaxPool];
  __shared__ float part[4][256];
  const int s = blockIdx.x / (a.tiles * a.tiles);
  const int t = blockIdx.x % (a.tiles * a.tiles);
  const int ti = t / a.tiles, tj = t % a.tiles;
  if (tj < ti) return;
  const int pn = pool_select(va, s, psh, ids, t == 0);
  __syncthreads();
  if (ti * 16 >= pn || tj * 16 >= pn) return;
  gram_tile<NST>(a, s, ti, tj, pn, ids, part);
}

// k_gram<1..N> (pool from the pool kernel: va null) and k_pool_gram<1..N>
// launchers indexed by dim / 64 - 1
using GramLaunch = void (*)(dim3, const VoteArgs*, const GramArgs&, hipStream_t);
template <int NST>
void launch_gram_n(dim3 g, const VoteArgs* va, const GramArgs& a, hipStream_t st) {
  if (va) hipLaunchKernelGGL(k_pool_gram<NST>, g, dim3(1024), 0, st, *va, a);
  else hipLaunchKernelGGL(k_gram<NST>, g, dim3(256), 0, st, a);
}
template <int... I>
const GramLaunch* gram_table(std::integer_sequence<int, I...>) {
  static const GramLaunch t[] = {&launch_gram_n<I + 1>...};
  return t;
}
template <int N>
const GramLaunch* gram_launchers() { return gram_table(std::make_integer_sequence<int, N>{}); }

// ---------------------------------------------------------------------------
// Append kernels
// ---------------------------------------------------------------------------
// Descriptor (Eq. memory_key): fp32 mean over the frame's raw last-layer tokens,
// heads flattened head-major, L2-normalised.  Also writes the frame offsets.
// Per (frame, layer): the mean raw key of every KV head becomes the frame's
// pooled key of that layer; the last shallow layer's means, flattened
// head-major and L2-normalised, are the unit descriptor (Eq. memory_key).
// Grid: (frames, layers).  Thread (slice s, 8-dim group v) sums tokens s, s + S,
// ... of its group with 16-byte loads (fp32, token order within the slice); the
// S slices are then added in slice order, so the sums are deterministic.
template <int D>
__global__ __launch_bounds__(256) void k_unit_means(AppendArgs a) {
  __shared__ float part[256 * 8];   // [slice][dim] partial sums (S * dim = 2048 floats)
  __shared__ float red[8];
  const int f = blockIdx.x, l = blockIdx.y;
  const int T = a.n_tokens, dim = a.Hk * D, G8 = dim / 8;
  const int S = 256 / G8;           // dim <= kMaxDescDim: G8 <= 128, S >= 2
  const int64_t nT = (int64_t)a.n_frames * T;
  const uint16_t* src = a.src[l];
  uint32_t amax = 0;   // largest |key element| (the bits of a non-negative float order as integers)
  if (threadIdx.x < S * G8) {
    const int v = threadIdx.x % G8, sl = threadIdx.x / G8;
    const int g = (8 * v) / D, e0 = (8 * v) % D;
    const uint16_t* p = src + ((int64_t)g * nT + (int64_t)f * T) * D + e0;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int t = sl;
    for (; t + 3 * S < T; t += 4 * S) {
      u32x4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = *reinterpret_cast<const u32x4*>(p + (int64_t)(t + u * S) * D);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          acc[2 * k] += bf16_lo(x[u][k]);
          acc[2 * k + 1] += bf16_hi(x[u][k]);
          amax = max(amax, max((x[u][k] << 16) & 0x7FFFFFFFu, x[u][k] & 0x7FFF0000u));
        }
    }
    for (; t < T; t += S) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(p + (int64_t)t * D);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc[2 * k] += bf16_lo(x[k]);
        acc[2 * k + 1] += bf16_hi(x[k]);
        amax = max(amax, max((x[k] << 16) & 0x7FFFFFFFu, x[k] & 0x7FFF0000u));
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) part[sl * dim + 8 * v + k] = acc[k];
  }
  amax = wave_max_u32(amax);
  if ((threadIdx.x & 63) == 0) atomicMax(a.dst.stats, amax);
  __syncthreads();
  float vals[4];
  float ss = 0.f;
  for (int k = 0; k < 4; ++k) {
    const int e = threadIdx.x + k * 256;
    vals[k] = 0.f;
    if (e < dim) {
      float acc = 0.f;
      for (int sl = 0; sl < S; ++sl) acc += part[sl * dim + e];
      vals[k] = acc / (float)T;
      ss = fmaf(vals[k], vals[k], ss);
    }
  }
  float* pooled = a.dst.pooled + ((a.frame0 + f) * a.L + l) * (int64_t)dim;
  for (int k = 0; k < 4; ++k) {
    const int e = threadIdx.x + k * 256;
    if (e < dim) pooled[e] = vals[k];
  }
  if (l != a.L - 1) return;  // the same for the whole block
  // deterministic block sum of squares
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = tot > 0.f ? 1.0f / sqrtf(tot) : 0.f;
  float* out = a.dst.desc + (a.frame0 + f) * (int64_t)dim;
  for (int k = 0; k < 4; ++k) {
    const int e = threadIdx.x + k * 256;
    if (e < dim) out[e] = tot > 0.f ? vals[k] * inv : 0.f;
  }
  if (threadIdx.x == 0) {
    a.dst.frame_off[a.frame0 + f + 1] = (int32_t)(a.row0 + (int64_t)(f + 1) * a.rows_per_frame);
    if (f == 0) a.dst.frame_off[a.frame0] = (int32_t)a.row0;
  }
}

// Raw rows: 16-byte copies into the arena, member counts = 1.
template <int D>
__global__ __launch_bounds__(256) void k_copy(AppendArgs a) {
  const int64_t nT = (int64_t)a.n_frames * a.n_tokens;
  const int64_t per_row = D / 8;
  const int64_t total = (int64_t)a.L * a.Hk * nT * per_row;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e8 = c % per_row;
    const int64_t rr = c / per_row;
    const int64_t r = rr % nT;
    const int64_t lg = rr / nT;
    const int g = (int)(lg % a.Hk), l = (int)(lg / a.Hk);
    const u32x4 v = *reinterpret_cast<const u32x4*>(a.src[l] + ((int64_t)g * nT + r) * D + 8 * e8);
    const int64_t drow = ((int64_t)l * a.Hk + g) * a.max_rows + a.row0 + r;
    *reinterpret_cast<u32x4*>(a.dst.keys + drow * D + 8 * e8) = v;
    if (e8 == 0) a.dst.counts[drow] = 1;
  }
}

// Per (frame, layer, KV head) k-means: farthest-point seeding from the frame
// mean, then n_iters Lloyd rounds on squared Euclidean distance in fp32.  One
// block of 16 waves per problem; wave w holds tokens 16w..16w+15 as an MFMA
// operand tile (bf16 16x16x32, fp32 accumulation).
//
// Exact products, bounded sums: the tokens are exact bf16, and every fp32
// centre is split exactly into three bf16 parts (c = c1 + c2 + c3), so every
// product in a dot product is exact and only the fp32 sums round (each addition
// off by at most 2^-23 relative, whatever the rounding mode of the matrix
// core).  An expanded distance |x|^2 + |y|^2 - 2 x.y then lies within a bound
// eps of the exact one (below), and wherever two candidates are closer than
// 2.5 eps the decision is taken again in the direct form sum_e (x_e - y_e)^2
// (fmaf in dimension order).  Every decision is therefore the exact one or the
// direct form's.
//
// Seeding: pick 0 is the token farthest from the frame mean (direct form).
// Each later pick is the token whose running minimum of expanded distances to
// the picks so far is largest (ties to the lower token); eps = 2^-24 max|x|^2
// (6D + 16).  Candidates near the maximum get their exact minimum over every
// pick so far.
//
// Assignment: per token the two smallest keys (ordered expanded distance, low 6
// bits = centre) over the centres, reduced over the 16 lanes of an MFMA row by
// DPP; eps = 2^-24 ((D + 8)(|x|^2 + max|c|^2) + 4 (D + 9) |x| max|c| + d) plus
// the key truncation.  Near ties are re-decided by one wave, one lane per centre.
//
// Update: the member sums are an MFMA contraction over the tokens (one-hot
// membership x tokens; exact products, a fixed summation order); a centre moves
// to sum / count, an empty centre stays.  The new centres are published as
// fp32 rows, squared norms and split MFMA operands.
// DPP move of a float / the two smallest of (k1, k2) and the partner's pair
template <int ctrl>
__device__ __forceinline__ float km_dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), ctrl, 0xF, 0xF, false));
}
template <int ctrl>
__device__ __forceinline__ void km_pair_min(uint32_t& k1, uint32_t& k2) {
  const uint32_t o1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k1, ctrl, 0xF, 0xF, false);
  const uint32_t o2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)k2, ctrl, 0xF, 0xF, false);
  k2 = min(max(k1, o1), min(k2, o2));
  k1 = min(k1, o1);
}

constexpr int kKmThreads = 1024;      // 16 waves: one 16-token tile per wave (T <= kMaxTokensCompress = 256)
constexpr int kKmMeanThreads = 256;   // threads of the frame-mean partial sums

template <int D>
struct KmLayout {
  static constexpr int KS = D / 32;        // k-steps of 32 dims
  static constexpr int Q = D / 8;          // 8-dim groups per row
  static constexpr int XW = D / 2 + 4;     // token row stride in 32-bit words (padded by 16 B)
  static constexpr int CS = D + 1;         // fp32 centre row stride in floats (conflict-free columns)
  // token rows, padded to whole 32-token MFMA k-steps
  __host__ __device__ static int rows(int T) { return (T + 31) / 32 * 32; }
  __host__ __device__ static size_t op_bytes(int C) { return (size_t)((C + 15) / 16) * 3 * KS * 64 * 16; }
  __host__ __device__ static size_t x_bytes(int T) { return (size_t)rows(T) * XW * 4; }
  // the centre rows also hold the frame mean's partial sums (kKmMeanThreads / Q slices of D)
  __host__ __device__ static size_t c_bytes(int C) {
    const size_t n = (size_t)C * CS, m = (size_t)8 * kKmMeanThreads;
    return (n > m ? n : m) * 4;
  }
  __host__ __device__ static size_t bytes(int T, int C) { return op_bytes(C) + x_bytes(T) + c_bytes(C); }
};

__device__ __forceinline__ float bf16f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Publishes the 8 dims 8q..8q+7 of centre c: the fp32 row (c < C), its exact
// three-part bf16 split as MFMA A operands, and (lane q == 0) the squared norm
// summed over the Q lanes of the centre in a fixed butterfly.  Every lane of
// the wave calls it (inactive items pass zeros and c >= C).
template <int D>
__device__ __forceinline__ void km_publish(int c, int q, int C, const float (&v)[8], float* cenf,
                                           u32x4* opA, float* cn) {
  using Lay = KmLayout<D>;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) ss = fmaf(v[k], v[k], ss);
  uint32_t w1[4], w2[4], w3[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint16_t p1[2], p2[2], p3[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float x = v[2 * k + h];
      p1[h] = bf16_rne(x);
      const float r1 = x - bf16f(p1[h]);
      p2[h] = bf16_rne(r1);
      p3[h] = bf16_rne(r1 - bf16f(p2[h]));
    }
    w1[k] = (uint32_t)p1[0] | ((uint32_t)p1[1] << 16);
    w2[k] = (uint32_t)p2[0] | ((uint32_t)p2[1] << 16);
    w3[k] = (uint32_t)p3[0] | ((uint32_t)p3[1] << 16);
  }
  if (c < (C + 15) / 16 * 16) {
    const int ct = c >> 4, ln = (c & 15) + 16 * (q & 3), ks = q >> 2;
    opA[((ct * 3 + 0) * Lay::KS + ks) * 64 + ln] = u32x4{w1[0], w1[1], w1[2], w1[3]};
    opA[((ct * 3 + 1) * Lay::KS + ks) * 64 + ln] = u32x4{w2[0], w2[1], w2[2], w2[3]};
    opA[((ct * 3 + 2) * Lay::KS + ks) * 64 + ln] = u32x4{w3[0], w3[1], w3[2], w3[3]};
  }
  if (c < C) {
#pragma unroll
    for (int k = 0; k < 8; ++k) cenf[c * Lay::CS + 8 * q + k] = v[k];
  }
  if (Lay::Q == 16) {   // the 16 lanes of the centre are one DPP row; lane q == 0 keeps its sum
    ss += km_dpp_f<0xB1>(ss);
    ss += km_dpp_f<0x4E>(ss);
    ss += km_dpp_f<0x124>(ss);
    ss += km_dpp_f<0x128>(ss);
  } else {
    ss += __shfl_xor(ss, 1);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 4);
  }
  if (q == 0 && c < C) cn[c] = ss;
}

// Direct squared distance sum_e (x_e - y_e)^2 (fmaf in dimension order) of a
// bf16 token row in LDS against another bf16 row, or against fp32 values read
// by `yv(e)`; 16 dims at a time are loaded ahead of the chain.
template <int D>
__device__ __forceinline__ float km_dist_rows(const uint32_t* xr, const uint32_t* yr) {
  float acc = 0.f;
#pragma unroll
  for (int c0 = 0; c0 < D / 8; c0 += 2) {
    u32x4 xa[2], ya[2];
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      xa[v] = *reinterpret_cast<const u32x4*>(xr + 4 * (c0 + v));
      ya[v] = *reinterpret_cast<const u32x4*>(yr + 4 * (c0 + v));
    }
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float d0 = bf16_lo(xa[v][k]) - bf16_lo(ya[v][k]);
        acc = fmaf(d0, d0, acc);
        const float d1 = bf16_hi(xa[v][k]) - bf16_hi(ya[v][k]);
        acc = fmaf(d1, d1, acc);
      }
  }
  return acc;
}
template <int D, class YV>
__device__ __forceinline__ float km_dist_row_f32(const uint32_t* xr, YV yv) {
  float acc = 0.f;
#pragma unroll
  for (int c0 = 0; c0 < D / 8; c0 += 2) {
    u32x4 xa[2];
    float y[16];
#pragma unroll
    for (int v = 0; v < 2; ++v) xa[v] = *reinterpret_cast<const u32x4*>(xr + 4 * (c0 + v));
#pragma unroll
    for (int e = 0; e < 16; ++e) y[e] = yv(8 * c0 + e);
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float d0 = bf16_lo(xa[v][k]) - y[8 * v + 2 * k];
        acc = fmaf(d0, d0, acc);
        const float d1 = bf16_hi(xa[v][k]) - y[8 * v + 2 * k + 1];
        acc = fmaf(d1, d1, acc);
      }
  }
  return acc;
}

// Exact (direct-form) minimum squared distance of token `tok` to the picks
// chosen[0..c-1], one lane per pick (c <= 64), reduced over the wave.  Kept out
// of line: it runs only near ties and would otherwise hold registers in the
// seeding loop.
template <int D>
__device__ __noinline__ float km_exact_min(const uint32_t* xs, int xw, const int* chosen, int tok, int c) {
  const int lane = threadIdx.x & 63;
  float m = lane < c ? km_dist_rows<D>(xs + tok * xw, xs + chosen[lane] * xw) : INFINITY;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) m = fminf(m, __shfl_xor(m, o));
  return m;
}

template <int D>
__global__ __launch_bounds__(kKmThreads) void k_kmeans(AppendArgs a) {
  using Lay = KmLayout<D>;
  constexpr int KS = Lay::KS, Q = Lay::Q, XW = Lay::XW, CS = Lay::CS;
  constexpr int NW = kKmThreads / 64;      // one 16-token tile per wave
  constexpr int SL = kKmMeanThreads / Q;   // token slices of the frame-mean partial sums
  constexpr int NDT = D / 16;              // dim tiles of the update
  constexpr int MAXS = kMaxTokensCompress / 32;
  extern __shared__ __align__(16) unsigned char km_dyn[];
  __shared__ float xn[kMaxTokensCompress];
  __shared__ __align__(16) int assign_[kMaxTokensCompress];
  __shared__ int rlist[kMaxTokensCompress];
  __shared__ float cn[kMaxCentroids];
  __shared__ int ccount[kMaxCentroids];
  __shared__ int chosen[kMaxCentroids];
  __shared__ float mu[D];
  __shared__ uint32_t shk[2][NW], shk2[2][NW];
  __shared__ int shi[2][NW];
  __shared__ float cval[kMaxTokensCompress];   // exact minima of near-tie candidates
  __shared__ float xnmax_sh;
  __shared__ int rcount, pick_sh;

  const int b = blockIdx.x;
  const int g = b % a.Hk, fl = b / a.Hk, l = fl % a.L, f = fl / a.L;
  const int T = a.n_tokens, C = min(a.n_centroids, T);
  const int nct = (C + 15) / 16, Tp = Lay::rows(T), ntt = (T + 15) / 16, nsteps = Tp / 32;
  const int64_t nT = (int64_t)a.n_frames * T;
  const uint16_t* src = a.src[l] + ((int64_t)g * nT + (int64_t)f * T) * D;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;

  u32x4* opA = reinterpret_cast<u32x4*>(km_dyn);
  uint32_t* xs = reinterpret_cast<uint32_t*>(km_dyn + Lay::op_bytes(C));
  float* cenf = reinterpret_cast<float*>(km_dyn + Lay::op_bytes(C) + Lay::x_bytes(T));

  // tokens -> LDS (bf16 rows, padded stride; rows T..Tp-1 zero); padded rows have no centre
  for (int i = t; i < Tp * Q; i += kKmThreads) {
    const int r = i / Q, v = i - r * Q;
    u32x4 x = {0u, 0u, 0u, 0u};
    if (r < T) x = *reinterpret_cast<const u32x4*>(src + (int64_t)r * D + 8 * v);
    *reinterpret_cast<u32x4*>(xs + r * XW + 4 * v) = x;
  }
  for (int r = t; r < kMaxTokensCompress; r += kKmThreads) assign_[r] = -1;
  if (t == 0) rcount = 0;
  __syncthreads();
  // frame mean: thread (slice s, group q) sums dims 8q..8q+7 over tokens s, s + SL, ...;
  // the slices' partial sums (staged in the centre rows, unused until seeding ends) are
  // then added in slice order.  Squared norms |x|^2 in dimension order (fmaf).
  if (t < kKmMeanThreads) {
    const int q = t % Q, s = t / Q;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int r = s; r < T; r += SL) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(xs + r * XW + 4 * q);
      const uint32_t ws[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
      for (int k = 0; k < 4; ++k) { acc[2 * k] += bf16_lo(ws[k]); acc[2 * k + 1] += bf16_hi(ws[k]); }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) cenf[s * D + 8 * q + k] = acc[k];
  } else if (t < kKmMeanThreads + kMaxTokensCompress) {
    const int r = t - kKmMeanThreads;
    float s2 = 0.f;
    if (r < T) {
#pragma unroll
      for (int v = 0; v < Q; ++v) {
        const u32x4 x = *reinterpret_cast<const u32x4*>(xs + r * XW + 4 * v);
        const uint32_t ws[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          s2 = fmaf(bf16_lo(ws[k]), bf16_lo(ws[k]), s2);
          s2 = fmaf(bf16_hi(ws[k]), bf16_hi(ws[k]), s2);
        }
      }
    }
    xn[r] = s2;
  }
  __syncthreads();
  if (t < D) {
    float acc = 0.f;
    for (int s = 0; s < SL; ++s) acc += cenf[s * D + t];
    mu[t] = acc / (float)T;
  } else if (t >= 64 * 4 && t < 64 * 5) {   // wave 4: the largest squared norm
    float m = 0.f;
    for (int r = lane; r < T; r += 64) m = fmaxf(m, xn[r]);
    const uint32_t mm = wave_max_u32(__float_as_uint(m));   // non-negative floats order as uint
    if (lane == 0) xnmax_sh = __uint_as_float(mm);
  }
  __syncthreads();

  // The wave's token tile (tokens 16w..16w+15) as MFMA A operands, kept for seeding
  // and assignment.  Output lane l holds tokens 16w + 4(l>>4) + j, j = 0..3; lane l
  // owns token tok_l = 16w + 4(l>>4) + (l&3) (four lanes per token, identical values).
  const bool has_tile = w < ntt;
  u32x4 A[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    A[ks] = has_tile ? *reinterpret_cast<const u32x4*>(xs + (16 * w + (lane & 15)) * XW + 16 * ks + 4 * (lane >> 4))
                     : u32x4{0u, 0u, 0u, 0u};
  const int my_tok = 16 * w + 4 * (lane >> 4) + (lane & 3);
  const bool tok_ok = has_tile && my_tok < T;
  const float my_xn = tok_ok ? xn[my_tok] : 0.f;
  const float xnmax = xnmax_sh;

  // ---- farthest-point seeding (pick 0 in the direct form, later picks from
  // MFMA dot products with the exact re-decision near ties)
  if (t < T) cval[t] = km_dist_row_f32<D>(xs + t * XW, [&](int e) { return mu[e]; });
  __syncthreads();
  float val = tok_ok ? cval[my_tok] : -INFINITY;
  bool avail = tok_ok;
  float my_min = INFINITY;
  const float band = 2.5f * 5.9604645e-8f * xnmax * (float)(6 * D + 16);
  for (int c = 0; c < C; ++c) {
    const int pb = c & 1;
    {
      // wave: largest value, its lowest token, the largest value of any other token
      const uint32_t o = avail ? ord_u32(val) : 0u;
      const uint32_t m1 = wave_max_u32(o);
      const uint64_t bm = __ballot(avail && o == m1);
      const int blane = bm ? __builtin_ctzll(bm) : 0;
      const int btok = 16 * w + 4 * (blane >> 4) + (blane & 3);
      const uint32_t m2 = wave_max_u32(avail && my_tok != btok ? o : 0u);
      if (lane == 0) {
        shk[pb][w] = m1;
        shk2[pb][w] = m2;
        shi[pb][w] = bm ? btok : INT_MAX;
      }
    }
    __syncthreads();
    // the waves' winners, lane i holding wave i's: the largest, its lowest token,
    // the largest of everything else (waves without a candidate hold zeros)
    uint32_t k1, k2;
    int pick;
    {
      const uint32_t a1 = lane < NW ? shk[pb][lane] : 0u, a2 = lane < NW ? shk2[pb][lane] : 0u;
      const int i1 = lane < NW ? shi[pb][lane] : INT_MAX;
      k1 = wave_max_u32(a1);
      pick = (int)wave_min_u32(a1 == k1 ? (uint32_t)i1 : (uint32_t)INT_MAX);
      k2 = wave_max_u32(max(i1 != pick ? a1 : 0u, a2));
    }
    if (c > 0 && k2 != 0u && ord_f32(k2) >= ord_f32(k1) - band) {
      // near tie: exact minima of the candidates over picks 0..c-1, one wave each
      if (t == 0) rcount = 0;
      __syncthreads();
      const float v1 = ord_f32(k1);
      if (avail && (lane >> 2 & 3) == 0 && val >= v1 - band) rlist[atomicAdd(&rcount, 1)] = my_tok;
      __syncthreads();
      const int ncand = rcount;
      for (int i = w; i < ncand; i += NW) {
        const float m = km_exact_min<D>(xs, XW, chosen, rlist[i], c);
        if (lane == 0) cval[i] = m;
      }
      __syncthreads();
      if (t == 0) {
        float bv = -INFINITY;
        int bt = INT_MAX;
        for (int i = 0; i < ncand; ++i) {
          const float m = cval[i];
          const int tok = rlist[i];
          if (m > bv || (m == bv && tok < bt)) { bv = m; bt = tok; }
        }
        pick_sh = bt;
      }
      __syncthreads();
      pick = pick_sh;
    }
    if (my_tok == pick) avail = false;
    if (t == 0) chosen[c] = pick;
    if (c == C - 1) break;
    if (has_tile) {   // wave-uniform: dot products with the pick
      u32x4 B[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        B[ks] = *reinterpret_cast<const u32x4*>(xs + pick * XW + 16 * ks + 4 * (lane >> 4));
      f32x4 h = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) h = mfma_bf16(A[ks], B[ks], h);
      const float xp = xn[pick];
      const int j = lane & 3;
      const float dot = j == 0 ? h[0] : j == 1 ? h[1] : j == 2 ? h[2] : h[3];
      my_min = fminf(my_min, fmaf(-2.f, dot, my_xn + xp));
    }
    val = my_min;
  }
  __syncthreads();
  // initial centres: the chosen tokens
  for (int i = t; i < nct * 16 * Q; i += kKmThreads) {
    const int c = i / Q, q = i - c * Q;
    float v[8];
    if (c < C) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(xs + chosen[c] * XW + 4 * q);
      const uint32_t ws[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
      for (int k = 0; k < 4; ++k) { v[2 * k] = bf16_lo(ws[k]); v[2 * k + 1] = bf16_hi(ws[k]); }
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = 0.f;
    }
    km_publish<D>(c, q, C, v, cenf, opA, cn);
  }
  if (t == 0) rcount = 0;
  __syncthreads();

  const int dt = w % NDT;
  for (int it = 0; it < a.n_iters; ++it) {
    // ---- assignment: MFMA dot products (A = the wave's 16 tokens, B = 16 centres),
    // expanded distances as keys (ordered distance, low 6 bits = centre), per token
    // the two smallest keys over the 16 lanes of an MFMA row (DPP), exact
    // re-decision near ties
    if (has_tile) {   // wave-uniform
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        A[ks] = *reinterpret_cast<const u32x4*>(xs + (16 * w + (lane & 15)) * XW + 16 * ks + 4 * (lane >> 4));
      float cmax = 0.f;
      for (int ct = 0; ct < nct; ++ct) {
        const int c = ct * 16 + (lane & 15);
        if (c < C) cmax = fmaxf(cmax, cn[c]);
      }
      cmax = fmaxf(cmax, km_dpp_f<0xB1>(cmax));
      cmax = fmaxf(cmax, km_dpp_f<0x4E>(cmax));
      cmax = fmaxf(cmax, km_dpp_f<0x124>(cmax));
      cmax = fmaxf(cmax, km_dpp_f<0x128>(cmax));
      float xv[4];
      uint32_t k1[4], k2[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xv[j] = xn[16 * w + 4 * (lane >> 4) + j];
        k1[j] = 0xFFFFFFFFu;
        k2[j] = 0xFFFFFFFFu;
      }
      for (int ct = 0; ct < nct; ++ct) {
        const int c = ct * 16 + (lane & 15);
        const float cc = c < C ? cn[c] : 0.f;
        f32x4 h = {0.f, 0.f, 0.f, 0.f}, m = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) h = mfma_bf16(A[ks], opA[((ct * 3 + 0) * KS + ks) * 64 + lane], h);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) m = mfma_bf16(A[ks], opA[((ct * 3 + 2) * KS + ks) * 64 + lane], m);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) m = mfma_bf16(A[ks], opA[((ct * 3 + 1) * KS + ks) * 64 + lane], m);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float d = fmaf(-2.f, h[j] + m[j], xv[j] + cc);
          const uint32_t kn = c < C ? ((ord_u32(d) & ~63u) | (uint32_t)c) : 0xFFFFFFFFu;
          if (kn < k1[j]) { k2[j] = k1[j]; k1[j] = kn; }
          else k2[j] = min(k2[j], kn);
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        km_pair_min<0xB1>(k1[j], k2[j]);
        km_pair_min<0x4E>(k1[j], k2[j]);
        km_pair_min<0x124>(k1[j], k2[j]);
        km_pair_min<0x128>(k1[j], k2[j]);
      }
      // lane (row r, j < 4) decides token 16w + 4r + j
      const int j = lane & 15, tok = 16 * w + 4 * (lane >> 4) + j;
      if (j < 4 && tok < T) {
        const uint32_t b1 = j == 0 ? k1[0] : j == 1 ? k1[1] : j == 2 ? k1[2] : k1[3];
        const uint32_t b2 = j == 0 ? k2[0] : j == 1 ? k2[1] : j == 2 ? k2[2] : k2[3];
        const float xx = j == 0 ? xv[0] : j == 1 ? xv[1] : j == 2 ? xv[2] : xv[3];
        assign_[tok] = b1 != 0xFFFFFFFFu ? (int)(b1 & 63u) : 0;
        if (b2 != 0xFFFFFFFFu) {
          const float d1 = ord_f32(b1 & ~63u), d2 = ord_f32(b2 & ~63u);
          const float eps = 5.9604645e-8f * ((float)(D + 8) * (xx + cmax) +
                                             (float)(4 * (D + 9)) * sqrtf(xx * cmax) + fabsf(d1));
          if (!(d2 - d1 > 2.5f * eps + 3.0517578e-5f * fabsf(d2))) rlist[atomicAdd(&rcount, 1)] = tok;
        }
      }
    }
    if (t < kMaxCentroids) ccount[t] = 0;
    __syncthreads();
    const int nref = rcount;
    for (int i = w; i < nref; i += NW) {   // direct form, lane = centre
      const int tok = rlist[i];
      float acc = INFINITY;
      if (lane < C) acc = km_dist_row_f32<D>(xs + tok * XW, [&](int e) { return cenf[lane * CS + e]; });
      int bi = lane < C ? lane : INT_MAX;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const float v2 = __shfl_xor(acc, o);
        const int i2 = __shfl_xor(bi, o);
        if (v2 < acc || (v2 == acc && i2 < bi)) { acc = v2; bi = i2; }
      }
      if (lane == 0) assign_[tok] = bi;
    }
    __syncthreads();
    if (t < T) atomicAdd(&ccount[assign_[t]], 1);
    if (t == 0) rcount = 0;
    __syncthreads();
    // ---- update: member sums as an MFMA contraction over the tokens (A = one-hot
    // membership of 16 centres, B = the wave's 16 dims of the tokens; exact products,
    // fixed summation order); mean = sum / count, an empty centre stays
      // the wave's dim tile of the tokens as MFMA B operands for the update (k = 32
      // tokens per step, column = dim); the tokens never change
      u32x4 xT[MAXS];
    #pragma unroll
      for (int st = 0; st < MAXS; ++st) {
        xT[st] = u32x4{0u, 0u, 0u, 0u};
        if (st >= nsteps) continue;   // wave-uniform
        const int dcol = dt * 16 + (lane & 15), t0 = 32 * st + 8 * (lane >> 4);
        uint32_t xb[4];
    #pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t w0 = xs[(t0 + 2 * k) * XW + (dcol >> 1)];
          const uint32_t w1 = xs[(t0 + 2 * k + 1) * XW + (dcol >> 1)];
          const uint32_t v0 = (dcol & 1) ? (w0 >> 16) : (w0 & 0xFFFFu);
          const uint32_t v1 = (dcol & 1) ? (w1 >> 16) : (w1 & 0xFFFFu);
          xb[k] = v0 | (v1 << 16);
        }
        xT[st] = u32x4{xb[0], xb[1], xb[2], xb[3]};
      }
    for (int ct = w / NDT; ct < nct; ct += NW / NDT) {   // wave-uniform
      const int crow = ct * 16 + (lane & 15);
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < MAXS; ++st) {
        if (st >= nsteps) continue;   // wave-uniform
        const int t0 = 32 * st + 8 * (lane >> 4);
        const int4 a0 = *reinterpret_cast<const int4*>(assign_ + t0);
        const int4 a1 = *reinterpret_cast<const int4*>(assign_ + t0 + 4);
        const u32x4 oh = {(a0.x == crow ? 0x3F80u : 0u) | (a0.y == crow ? 0x3F800000u : 0u),
                          (a0.z == crow ? 0x3F80u : 0u) | (a0.w == crow ? 0x3F800000u : 0u),
                          (a1.x == crow ? 0x3F80u : 0u) | (a1.y == crow ? 0x3F800000u : 0u),
                          (a1.z == crow ? 0x3F80u : 0u) | (a1.w == crow ? 0x3F800000u : 0u)};
        acc = mfma_bf16(oh, xT[st], acc);
      }
      const int dcol = dt * 16 + (lane & 15);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = ct * 16 + 4 * (lane >> 4) + j;
        if (c < C) {
          const int n = ccount[c];
          if (n > 0) cenf[c * CS + dcol] = acc[j] / (float)n;
        }
      }
    }
    __syncthreads();
    for (int i = t; i < nct * 16 * Q; i += kKmThreads) {
      const int c = i / Q, q = i - c * Q;
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = c < C ? cenf[c * CS + 8 * q + k] : 0.f;
      km_publish<D>(c, q, C, v, cenf, opA, cn);
    }
    __syncthreads();
  }
  const int64_t drow0 = ((int64_t)l * a.Hk + g) * a.max_rows + a.row0 + (int64_t)f * C;
  for (int i = t; i < C * D; i += kKmThreads) {
    const int c = i / D, e = i - c * D;
    a.dst.keys[(drow0 + c) * D + e] = bf16_rne(cenf[c * CS + e]);
  }
  for (int c = t; c < C; c += kKmThreads) a.dst.counts[drow0 + c] = a.n_iters > 0 ? ccount[c] : 0;
}

// ---------------------------------------------------------------------------
// Pooled shallow Q-K ranking: keys pooled per unit at append (k_unit_means),
// scored against the question's pooled query weights, top-K units.
// ---------------------------------------------------------------------------
struct PoolQArgs {
  int Hq, Hk, G, L, first;
  const uint16_t* q[128];   // (stream, layer) pairs first .. first + 127
  int nq[kMaxStreams];
  float* w;                 // [pairs][H_kv][D]
};

// w[pair][g][e] = (sum over the group's heads and the question's tokens of q) /
// (n_q L H_q sqrt(D)): the weights whose dot product with a unit's pooled keys
// is its pooled score.  Grid: pairs x H_kv; 8 token groups of D threads, each
// summing every 8th (head, token) row with four loads in flight; the groups'
// partial sums are added in a fixed order.
constexpr int kPoolQGroups = 8;
template <int D>
__global__ __launch_bounds__(kPoolQGroups * D) void k_pool_query(PoolQArgs a) {
  __shared__ float part[kPoolQGroups][D];
  const int pl = blockIdx.x / a.Hk, g = blockIdx.x % a.Hk;
  const int pair = a.first + pl, s = pair / a.L;
  const int nq = a.nq[s], tg = threadIdx.x / D, e = threadIdx.x % D;
  const uint16_t* q = a.q[pl] + (size_t)g * a.G * nq * D + e;   // rows of the group's heads
  const int rows = a.G * nq;
  float acc = 0.f;
  int r = tg;
  for (; r + 3 * kPoolQGroups < rows; r += 4 * kPoolQGroups) {
    uint16_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = q[(size_t)(r + u * kPoolQGroups) * D];
#pragma unroll
    for (int u = 0; u < 4; ++u) acc += __uint_as_float((uint32_t)v[u] << 16);
  }
  for (; r < rows; r += kPoolQGroups) acc += __uint_as_float((uint32_t)q[(size_t)r * D] << 16);
  part[tg][e] = acc;
  __syncthreads();
  if (tg != 0) return;
  float x = part[0][e];
  for (int k = 1; k < kPoolQGroups; ++k) x += part[k][e];
  const float scale = 1.0f / ((float)nq * (float)a.L * (float)a.Hq * sqrtf((float)D));
  a.w[((size_t)pair * a.Hk + g) * D + e] = x * scale;
}

struct PoolScoreArgs {
  int n4;                           // float4 per unit: L H_kv D / 4
  const int32_t* count;             // null, or a device count that caps F[0] (one stream)
  int64_t F[kMaxStreams];
  const float4* pooled[kMaxStreams];
  const float4* w;                  // [S][n4]
  float* scores;                    // [S][f_max]
  int64_t f_max;
};

// One wave per unit: a fixed strided split over the lanes and a fixed
// butterfly, so a unit's score does not depend on the launch.
__global__ __launch_bounds__(256) void k_pool_score(PoolScoreArgs a) {
  const int s = blockIdx.y, lane = threadIdx.x & (kWave - 1);
  const int64_t f = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t F = a.count ? min<int64_t>(a.F[s], *a.count) : a.F[s];
  if (f >= F) return;   // whole waves leave together
  const float4* k = a.pooled[s] + f * a.n4;
  const float4* w = a.w + (size_t)s * a.n4;
  float acc = 0.f;
  for (int i = lane; i < a.n4; i += kWave) {
    const float4 x = k[i], y = w[i];
    acc = fmaf(x.x, y.x, acc);
    acc = fmaf(x.y, y.y, acc);
    acc = fmaf(x.z, y.z, acc);
    acc = fmaf(x.w, y.w, acc);
  }
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) a.scores[(size_t)s * a.f_max + f] = acc;
}

struct PoolSelectArgs {
  int n_select;
  const int32_t* count;             // null, or a device count that caps F[0] (one stream)
  const int64_t* span;              // null, or [F][2] first/last frame of each unit
  int64_t* out_first;               // with span: [S][n_select]
  int64_t* out_last;
  int64_t F[kMaxStreams];
  int64_t frame0[kMaxStreams];      // added to the window-relative ids
  const float* scores;              // [S][f_max]
  int64_t f_max;
  int64_t* out_ids;                 // [S][n_select]
  float* out_scores;
  int32_t* out_n;
};

// Top n_select units of a stream by (score desc, unit asc): a radix cut over
// the composite keys (scores staged in LDS when they fit), then ranks by
// counting.
constexpr int kPoolLds = 8192;
__global__ __launch_bounds__(1024) void k_pool_select(PoolSelectArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t res[4];
  __shared__ uint64_t sel[kMaxSelect];
  __shared__ uint32_t nsel;
  const int s = blockIdx.x;
  const int64_t F = a.count ? min<int64_t>(a.F[s], *a.count) : a.F[s];
  const int K = (int)min<int64_t>(a.n_select, F);
  __shared__ float lsc[kPoolLds];
  const float* gsc = a.scores + (size_t)s * a.f_max;
  const bool in_lds = F <= kPoolLds;
  if (in_lds)
    for (int i = threadIdx.x; i < F; i += blockDim.x) lsc[i] = gsc[i];
  const float* sc = in_lds ? lsc : gsc;
  auto key = [&](int i) -> uint64_t { return mk_key(ord_u32(sc[i] + 0.0f), (uint32_t)i); };
  if (threadIdx.x == 0) nsel = 0;
  __syncthreads();
  uint64_t cut = 0;
  if (K > 0 && K < F) cut = radix_select_u64(key, (int)F, (uint32_t)K, hist, res);
  __syncthreads();
  for (int i = threadIdx.x; i < F && K > 0; i += blockDim.x) {
    const uint64_t k = key(i);
    if (k >= cut) {
      const uint32_t slot = atomicAdd(&nsel, 1u);
      if (slot < (uint32_t)kMaxSelect) sel[slot] = k;
    }
  }
  __syncthreads();
  // each selected key goes to its rank (the number of larger selected keys)
  int64_t* ids = a.out_ids + (size_t)s * a.n_select;
  float* scs = a.out_scores + (size_t)s * a.n_select;
  if (threadIdx.x < K) {
    const uint64_t k = sel[threadIdx.x];
    int rank = 0;
    for (int m = 0; m < K; ++m) rank += sel[m] > k;
    ids[rank] = (int64_t)key_row(k) + a.frame0[s];
    scs[rank] = key_score(k);
    if (a.span) {
      a.out_first[(size_t)s * a.n_select + rank] = a.span[2 * (size_t)key_row(k)];
      a.out_last[(size_t)s * a.n_select + rank] = a.span[2 * (size_t)key_row(k) + 1];
    }
  }
  for (int i = K + threadIdx.x; i < a.n_select; i += blockDim.x) {
    ids[i] = -1;
    scs[i] = 0.f;
    if (a.span) {
      a.out_first[(size_t)s * a.n_select + i] = -1;
      a.out_last[(size_t)s * a.n_select + i] = -1;
    }
  }
  if (threadIdx.x == 0) a.out_n[s] = K;
}

// ---------------------------------------------------------------------------
// Long-history compression (Eq. optional_long_memory_clustering and Eq.
// optional_long_memory_representative).  k_cluster_assign walks the leaving
// units in temporal order in one block (each decision needs the centroid the
// previous one left); k_cluster_reps then replays the recorded assignments for
// every element of the representative keys in parallel.
// ---------------------------------------------------------------------------

__global__ void k_zero32(int32_t* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

// Sum over a 256-thread block, the same order every time.
__device__ float block_sum256(float v, float* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(256) void k_cluster_assign(AbsorbArgs a) {
  __shared__ float red[4];
  const int dim = a.Hk * a.D;   // at most 1024: four elements per thread
  int nc = a.cl.state[0], ovf = a.cl.state[1];
  int n = nc > 0 ? a.cl.sizes[nc - 1] : 0;
  float c[4] = {0.f, 0.f, 0.f, 0.f};
  if (nc > 0)
    for (int k = 0; k < 4; ++k) {
      const int e = threadIdx.x + 256 * k;
      if (e < dim) c[k] = a.cl.centroids[(size_t)(nc - 1) * dim + e];
    }
  for (int u = 0; u < a.n_units; ++u) {
    const int64_t t = a.f_lo + u;
    float kv[4] = {0.f, 0.f, 0.f, 0.f};
    float part = 0.f;
    for (int k = 0; k < 4; ++k) {
      const int e = threadIdx.x + 256 * k;
      if (e < dim) kv[k] = a.desc[(int64_t)u * dim + e];
      part = fmaf(kv[k], c[k], part);
    }
    bool join = false;
    if (nc > 0) {
      const float dot = block_sum256(part, red);
      join = dot >= a.tau;
      if (!join && nc == a.max_clusters) {
        join = true;
        ovf = 1;
      }
    }
    if (join) {
      // c <- Norm((n c + k) / (n + 1))
      float z[4], zz = 0.f;
      for (int k = 0; k < 4; ++k) {
        z[k] = ((float)n * c[k] + kv[k]) / (float)(n + 1);
        zz = fmaf(z[k], z[k], zz);
      }
      const float nrm = sqrtf(block_sum256(zz, red));
      for (int k = 0; k < 4; ++k) c[k] = nrm > 0.f ? z[k] / nrm : z[k];
      if (threadIdx.x == 0) {
        a.assign[2 * u] = nc - 1;
        a.assign[2 * u + 1] = n;
        a.cl.span[2 * (size_t)(nc - 1) + 1] = t;
      }
      ++n;
    } else {
      if (nc > 0) {
        for (int k = 0; k < 4; ++k) {
          const int e = threadIdx.x + 256 * k;
          if (e < dim) a.cl.centroids[(size_t)(nc - 1) * dim + e] = c[k];
        }
        if (threadIdx.x == 0) a.cl.sizes[nc - 1] = n;
      }
      for (int k = 0; k < 4; ++k) c[k] = kv[k];
      if (threadIdx.x == 0) {
        a.assign[2 * u] = nc;
        a.assign[2 * u + 1] = 0;
        a.cl.span[2 * (size_t)nc] = t;
        a.cl.span[2 * (size_t)nc + 1] = t;
      }
      n = 1;
      ++nc;
    }
  }
  if (nc > 0) {
    for (int k = 0; k < 4; ++k) {
      const int e = threadIdx.x + 256 * k;
      if (e < dim) a.cl.centroids[(size_t)(nc - 1) * dim + e] = c[k];
    }
  }
  if (threadIdx.x == 0) {
    if (nc > 0) a.cl.sizes[nc - 1] = n;
    a.cl.state[0] = nc;
    a.cl.state[1] = ovf;
  }
}

// One thread per element of a representative ([L][H_kv][R][D]): replays the
// call's units in order, (n rep + K) / (n + 1) with the recorded n.
__global__ __launch_bounds__(256) void k_cluster_reps(AbsorbArgs a) {
  const int64_t E = (int64_t)a.L * a.Hk * a.R * a.D;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const int d = (int)(e % a.D);
  const int64_t lgr = e / a.D;
  const int r = (int)(lgr % a.R);
  const int64_t lg = lgr / a.R;   // l * H_kv + g
  const uint16_t* src = a.keys + (lg * a.max_rows + a.row_lo + r) * a.D + d;
  int cur = -1;
  float v = 0.f;
  for (int u = 0; u < a.n_units; ++u) {
    const int j = a.assign[2 * u], nb = a.assign[2 * u + 1];
    if (j != cur) {
      if (cur >= 0) a.cl.reps[(size_t)cur * E + e] = v;
      cur = j;
      v = nb > 0 ? a.cl.reps[(size_t)j * E + e] : 0.f;
    }
    const float k = __uint_as_float((uint32_t)src[(int64_t)u * a.R * a.D] << 16);
    v = nb == 0 ? k : ((float)nb * v + k) / (float)(nb + 1);
  }
  if (cur >= 0) a.cl.reps[(size_t)cur * E + e] = v;
}

// ---------------------------------------------------------------------------
// Index compaction (the memory side of long-history compression)
// ---------------------------------------------------------------------------
// Copies len units from unit src to unit dst in each of n_seg segments
// (seg_stride units apart).  The host cuts a move into passes of at most the
// shift, so a launch's source and destination ranges never overlap and its
// copies may run in any order; the passes follow one another on the stream.
__global__ __launch_bounds__(256) void k_move16(u32x4* base, int64_t seg_stride, int n_seg, int64_t src,
                                                int64_t dst, int64_t len) {
  const int64_t total = len * n_seg;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t sg = i / len, e = i - sg * len;
    u32x4* b = base + sg * seg_stride;
    b[dst + e] = b[src + e];
  }
}

// The same for 4-byte words, subtracting `sub` from each (row offsets are
// rebased as they move; 0 for data).
__global__ __launch_bounds__(256) void k_move4(uint32_t* base, int64_t seg_stride, int n_seg, int64_t src,
                                               int64_t dst, int64_t len, uint32_t sub) {
  const int64_t total = len * n_seg;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t sg = i / len, e = i - sg * len;
    uint32_t* b = base + sg * seg_stride;
    b[dst + e] = b[src + e] - sub;
  }
}

// ---------------------------------------------------------------------------
// k_evidence: Eq. selected_evidence plus deduplication and temporal order.
// One block per stream: the recent window and every selected frame's
// neighbourhood are laid out as candidate slots (missing ones as a sentinel),
// sorted ascending in LDS, and the distinct values compacted in order.
// ---------------------------------------------------------------------------
// Items sort by their position in the stream: a detailed unit t at t, a
// long-term cluster at its first member unit.  Key = position << 32 | kind << 31
// | id (a position below 2^31, ids below 2^31); stored inverted (~key) so that
// a descending sort gives temporal order and an empty slot (0) sorts last.
__device__ __forceinline__ uint64_t evidence_key(int64_t pos, int kind, int64_t id) {
  return ~(((uint64_t)pos << 32) | ((uint64_t)kind << 31) | (uint64_t)id);
}

__global__ __launch_bounds__(256) void k_evidence(EvidenceArgs a) {
  __shared__ uint64_t buf[kMaxEvidence];
  __shared__ int scan_sh[17];
  const int s = blockIdx.x;
  const int64_t T = a.T[s], lo = a.lo[s];
  const int64_t r0 = max(lo, T > a.n_recent ? T - a.n_recent : (int64_t)0);
  const int nrec = (int)max((int64_t)0, T - r0);
  const int span = a.n_before + 1 + a.n_after;
  const int ndet = nrec + (a.retrieved ? a.n_select * span : 0);
  const int ncl = (a.retrieved && a.cl_span[s]) ? a.k_clusters : 0;
  const int total = ndet + ncl;
  const int P = pow2_ceil(max(total, 2));
  const int32_t n_cl = ncl > 0 ? *a.cl_count[s] : 0;
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    uint64_t key = 0;
    if (i < nrec) {
      key = evidence_key(r0 + i, 0, r0 + i);
    } else if (i < ndet) {
      const int j = i - nrec, slot = j / span, off = j % span - a.n_before;
      const int64_t t = a.frame_ids[(size_t)s * a.n_select + slot];
      // detailed units only: neighbours inside long-term clusters are not units any more
      if (t >= 0 && t < T && t + off >= lo && t + off < T) key = evidence_key(t + off, 0, t + off);
    } else if (i < total) {
      const int64_t c = a.cluster_ids[(size_t)s * a.k_clusters + (i - ndet)];
      if (c >= 0 && c < n_cl) key = evidence_key(a.cl_span[s][2 * c], 1, c);
    }
    buf[i] = key;
  }
  __syncthreads();
  bitonic_desc_u64(buf, P);
  int64_t* out = a.units + (size_t)s * a.max_units;
  int32_t* kinds = a.kinds ? a.kinds + (size_t)s * a.max_units : nullptr;
  int base = 0;
  for (int b0 = 0; b0 < P; b0 += blockDim.x) {
    const int i = b0 + threadIdx.x;
    const bool keep = i < P && buf[i] != 0 && (i == 0 || buf[i] != buf[i - 1]);
    int tot;
    const int pre = block_excl_scan(keep ? 1 : 0, scan_sh, tot);
    if (keep) {
      const uint64_t key = ~buf[i];
      out[base + pre] = (int64_t)(key & 0x7FFFFFFFu);
      if (kinds) kinds[base + pre] = (int32_t)((key >> 31) & 1u);
    }
    base += tot;
  }
  for (int i = base + threadIdx.x; i < a.max_units; i += blockDim.x) {
    out[i] = -1;
    if (kinds) kinds[i] = -1;
  }
  if (threadIdx.x == 0) a.n_units[s] = base;
}

inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

template <int D>
hipError_t append_impl(const AppendArgs& a, bool compress, hipStream_t st) {
  hipLaunchKernelGGL(k_unit_means<D>, dim3(a.n_frames, a.L), dim3(256), 0, st, a);
  if (compress) {
    const int C = std::min(a.n_centroids, a.n_tokens);
    const size_t lds = KmLayout<D>::bytes(a.n_tokens, C);
    // the largest layout the API admits (n_tokens <= 256, n_centroids <= 64) fits in 160 KB
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_kmeans<D>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)KmLayout<D>::bytes(kMaxTokensCompress, kMaxCentroids));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_kmeans<D>, dim3(a.n_frames * a.L * a.Hk), dim3(kKmThreads), lds, st, a);
  } else {
    const int64_t total = (int64_t)a.L * a.Hk * a.n_frames * a.n_tokens * (D / 8);
    const int grid = (int)std::min<int64_t>(cdiv(total, 256), 8192);
    hipLaunchKernelGGL(k_copy<D>, dim3(grid), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Retrieval orchestration
// ---------------------------------------------------------------------------
ScoreArgs make_score_args(const RetrievePlan& p, int kind) {
  ScoreArgs a{};
  a.L = p.L; a.Hq = p.Hq; a.Hk = p.Hk; a.G = p.G; a.NL = p.NL; a.ngs = p.ngs;
  a.head_mode = p.head_mode;
  a.S = p.S;
  a.chunk = kind == K_SAMPLE ? p.samp_chunk : p.chunk_rows;
  a.qB = reinterpret_cast<const u32x4*>(p.qB);
  int items = 0;
  for (int s = 0; s < p.S; ++s) {
    a.keys[s] = p.st[s].keys;
    a.stride[s] = p.st[s].row_stride;
    a.n[s] = p.st[s].n;
    a.units[s] = kind == K_SAMPLE ? p.st[s].m : p.st[s].n;
    a.samp_step[s] = p.st[s].m > 0 ? (int64_t)(((unsigned __int128)p.st[s].n << 32) / (unsigned)p.st[s].m) : 0;
    a.item_base[s] = items;
    items += p.L * p.ngs * cdiv(a.units[s], a.chunk);
  }
  a.item_base[p.S] = items;
  a.total_items = items;
  int64_t tiles = 0;
  for (int s = 0; s < p.S; ++s) {
    a.tile_base[s] = tiles;
    a.ntile[s] = cdiv(p.st[s].n, kTile);
    tiles += (int64_t)p.L * p.Hk * a.ntile[s];
  }
  a.tile_base[p.S] = tiles;
  a.samp = p.samp; a.samp_stride = p.m_max;
  a.tau = p.tau; a.cnt = p.cnt; a.cand = p.cand; a.cap = p.cap;
  a.only_list = -1; a.full = nullptr; a.row0 = 0;
  a.sgroup = kStreamGroupMax;
  a.xcd_weights = 0;
  a.dyn_tiles = 0;
  a.dyn_chunk = kDynChunk;
  a.dyn_ctr = p.dyn_ctr;
  return a;
}

// Blocks of the streaming pass: all resident at once, so that every wave takes
// one contiguous share of the tiles; two resident blocks (8 waves) per CU.
// Measured on gfx950, reads with about
// 32 KiB of nontemporal loads in flight per CU reach 7.1 TB/s with 4 to 8 waves
// per CU and only 6.8 to 6.9 TB/s with 12 to 16, and the streaming pass went
// from 425.6 us (4 blocks per CU) to 410.4 us on the 1-hour index.
constexpr int kStreamBlocksPerCU = 2;

// Cached per device (one atomic slot each: concurrent first calls compute the
// same value, and no call reads a half-written one).
constexpr int kMaxDevices = 64;

// KIND 0: k_stream, 1: k_stream_hm, 2: k_stream_hp<D, HK>.
template <int D, int KIND, int HK = 1>
int stream_grid() {
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  std::atomic<int>& slot = cache[dev % kMaxDevices];
  int grid = slot.load(std::memory_order_relaxed);
  if (grid == 0) {
    int cus = 256, per_cu = 0;
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const void* fn = KIND == 0 ? reinterpret_cast<const void*>(k_stream<D>)
                     : KIND == 1 ? reinterpret_cast<const void*>(k_stream_hm<D>)
                                 : reinterpret_cast<const void*>(k_stream_hp<D, HK>);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, 0) != hipSuccess || per_cu < 1)
      per_cu = 1;
    grid = std::min(per_cu, kStreamBlocksPerCU) * std::max(cus, 1);
    slot.store(grid, std::memory_order_relaxed);
  }
  return grid;
}

// Blocks per XCD group of the streaming pass: the largest power of two up to
// kStreamGroupMax whose group range spans at most three average segments.
int stream_group(int grid, int nseg) {
  int g = kStreamGroupMax;
  while (g > 1 && (int64_t)g * nseg > 3 * (int64_t)grid) g >>= 1;
  return g;
}

template <int D, int KIND>
void launch_score(const ScoreArgs& a, int head_mode, int max_grid, hipStream_t st) {
  if (a.total_items == 0) return;
  const int grid = std::min(a.total_items, max_grid);
  if (head_mode == 0) hipLaunchKernelGGL((k_score<D, KIND>), dim3(grid), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((k_score_hm<D, KIND>), dim3(grid), dim3(256), 0, st, a);
}

// The head-mode-1 probability streaming pass for the layer's KV-head count
// (H_kv * d <= 512: every B tile stays in registers).
template <int D, int HK>
void launch_stream_hp_hk(ScoreArgs a, const RetrievePlan& p, int64_t tiles, int cus, hipStream_t st) {
  const int grid = (int)std::min<int64_t>(stream_grid<D, 2, HK>(), std::max<int64_t>(1, tiles / 16));
  int nseg = 0;   // (stream, layer) segments with rows
  for (int s = 0; s < p.S; ++s) nseg += a.ntile[s] > 0 ? p.L : 0;
  a.sgroup = stream_group(grid, nseg);
  a.xcd_weights = cus == 256;
  hipLaunchKernelGGL((k_stream_hp<D, HK>), dim3(grid), dim3(256), 0, st, a);
}

template <int D>
hipError_t launch_stream_hp(const ScoreArgs& a, const RetrievePlan& p, int64_t tiles, int cus, hipStream_t st) {
  switch (p.Hk) {
    case 1: launch_stream_hp_hk<D, 1>(a, p, tiles, cus, st); return hipSuccess;
    case 2: launch_stream_hp_hk<D, 2>(a, p, tiles, cus, st); return hipSuccess;
    case 4: launch_stream_hp_hk<D, 4>(a, p, tiles, cus, st); return hipSuccess;
    case 8:
      if (D * 8 <= 512) { launch_stream_hp_hk<D, (D * 8 <= 512 ? 8 : 4)>(a, p, tiles, cus, st); return hipSuccess; }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t retrieve_impl(RetrievePlan& p, hipStream_t st) {
  // 1. query prep, fused with 2., the sample scores, in k_prep_sample (head
  // mode 0) when its blocks fit one round: at most one per CU (104 VGPRs at
  // d = 128).  Measured: 1-hour index -3 us, 10-minute -2 us, compressed
  // -1 us per call; on the 16-stream batch (about 800 blocks) the two kernels
  // are faster.
  const int pairs = p.S * p.L;
  PsArgs ps{};
  int ps_blocks = 0;
  for (int s = 0; s < p.S; ++s) {
    ps.blk_base[s] = ps_blocks;
    ps.spg[s] = std::max(1, cdiv(cdiv(p.st[s].m, kTile), kPsTiles));   // every group forms its B tile
    ps_blocks += p.L * p.Hk * ps.spg[s];
  }
  ps.blk_base[p.S] = ps_blocks;
  int cus = 256, dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  // head mode 1 with attention probabilities keeps every head's logits: its
  // prep and sample are head mode 0's (one sampled list per head)
  const int prep_hm = p.hm_prob ? 0 : p.head_mode;
  const int lists = p.S * p.NL;
  // prep, sample and cut-off in one launch (k_prep_thresh) when every list's
  // block fits one round and the sample is at most 2,048 rows: every block
  // gathers its group's whole sample, which pays while that is short (A/B on
  // one box: 10-minute index 110.9 -> 110.2 us per call, m = 1,072; compressed
  // 58.5 -> 56.3 us, m = 262) but not at the 1-hour index's 3,216 rows
  // (450.2 -> 456.3 us)
  const bool pt = D == 128 && p.head_mode == 0 && !p.hm_prob && pairs <= 128 && lists <= cus && p.m_max <= 2048;
  ps.xcd_map = cus == 256 && ps_blocks % 8 == 0;
  const bool fused = !pt && prep_hm == 0 && pairs <= 128 && ps_blocks <= cus;
  int nq_max = 0;
  for (int s = 0; s < p.S; ++s) nq_max = std::max(nq_max, p.st[s].nq);
  const bool hm_prep = prep_hm == 1 && pairs <= 128 && p.Hk <= 8 && p.G * nq_max <= kHmPrepTerms;
  PrepArgs pa_fused{};
  for (int first = 0; first < pairs; first += 128) {
    PrepArgs a{};
    a.Hq = p.Hq; a.Hk = p.Hk; a.G = p.G; a.L = p.L; a.head_mode = prep_hm; a.first = first;
    const int cnt = std::min(128, pairs - first);
    for (int i = 0; i < cnt; ++i) {
      const int pr = first + i;
      a.q[i] = p.st[pr / p.L].q[pr % p.L];
    }
    for (int s = 0; s < p.S; ++s) { a.nq[s] = p.st[s].nq; a.qscale[s] = p.st[s].qscale; }
    a.qB = reinterpret_cast<u32x4*>(p.qB);
    a.qcol = p.qcol;
    if (fused || pt || hm_prep)
      pa_fused = a;
    else
      hipLaunchKernelGGL(k_prep<D>, dim3(cnt * p.Hk), dim3(8 * D), 0, st, a);
  }
  ListArgs la{};
  la.NL = p.NL; la.S = p.S; la.cap = p.cap; la.k_max = p.k_max; la.top_k = p.top_k;
  for (int s = 0; s < p.S; ++s) {
    la.m[s] = p.st[s].m; la.r[s] = p.st[s].r; la.kk[s] = p.st[s].kk; la.n[s] = p.st[s].n;
    la.f[s] = p.st[s].f; la.rpf[s] = p.st[s].rpf; la.frame_off[s] = p.st[s].frame_off;
    la.row0[s] = p.st[s].row0;
    la.kmax[s] = p.st[s].kmax;
  }
  la.samp = p.samp; la.samp_stride = p.m_max; la.tau = p.tau; la.cnt = p.cnt;
  la.cand = p.cand;
  la.L = p.L; la.Hq = p.Hq; la.Hk = p.Hk; la.G = p.G; la.head_mode = p.head_mode;
  la.qB = reinterpret_cast<const u32x4*>(p.qB);
  for (int s = 0; s < p.S; ++s) { la.keys[s] = p.st[s].keys; la.stride[s] = p.st[s].row_stride; }
  la.dbg_pos = p.dbg_topk_pos; la.dbg_score = p.dbg_topk_score; la.dbg_stats = p.dbg_list_stats;
  la.f_max = p.f_max; la.votes_g = p.votes; la.massfx_g = p.massfx; la.sexp = p.sexp; la.qcol = p.qcol;
  la.dyn_ctr = p.dyn_ctr;
  la.score_mode = p.score_mode; la.hm_prob = p.hm_prob ? 1 : 0; la.NLs = p.NLs;
  la.below = p.below; la.lhat = p.lhat; la.cand_sc = p.cand_sc; la.left_max = p.left_max;
  la.cand_lse = p.cand_lse;
  // 2. sample scores, 3. thresholds
  if (pt) {
    PtArgs t{};
    t.NL = p.NL; t.L = p.L; t.Hq = p.Hq; t.Hk = p.Hk; t.G = p.G; t.f_max = p.f_max;
    t.xcd_map = cus == 256 && lists % 8 == 0 && (lists / 8) % p.G == 0;
    for (int s = 0; s < p.S; ++s) {
      t.keys[s] = p.st[s].keys;
      t.stride[s] = p.st[s].row_stride;
      t.n[s] = p.st[s].n;
      t.m[s] = p.st[s].m;
      t.r[s] = p.st[s].r;
      t.f[s] = p.st[s].f;
      t.samp_step[s] = p.st[s].m > 0 ? (int64_t)(((unsigned __int128)p.st[s].n << 32) / (unsigned)p.st[s].m) : 0;
    }
    t.tau = p.tau; t.cnt = p.cnt; t.below = p.below; t.dyn_ctr = p.dyn_ctr;
    t.votes_g = p.votes; t.massfx_g = p.massfx;
    hipLaunchKernelGGL(k_prep_thresh<2>, dim3(lists), dim3(1024), 0, st, pa_fused, t);
  } else if (prep_hm == 0) {
    ScoreArgs a = make_score_args(p, K_SAMPLE);
    a.NL = p.NLs;        // sampled lists: one per (layer, query head)
    a.head_mode = 0;
    int64_t tiles = 0;   // sample tiles of every (stream, layer, KV head)
    for (int s = 0; s < p.S; ++s) {
      a.tile_base[s] = tiles;
      a.ntile[s] = cdiv(p.st[s].m, kTile);
      tiles += (int64_t)p.L * p.Hk * a.ntile[s];
    }
    a.tile_base[p.S] = tiles;
    if (fused) {
      hipLaunchKernelGGL(k_prep_sample<D>, dim3(ps_blocks), dim3(8 * D), 0, st, pa_fused, a, ps);
    } else if (tiles > 0) {
      const int grid = (int)std::min<int64_t>(stream_grid<D, 0>(), std::max<int64_t>(1, tiles / 4));
      hipLaunchKernelGGL(k_sample<D>, dim3(grid), dim3(256), 0, st, a);
    }
  } else if (hm_prep) {
    ScoreArgs a = make_score_args(p, K_SAMPLE);
    if (a.total_items > 0)
      hipLaunchKernelGGL(k_score_hm_prep<D>, dim3(std::min(a.total_items, 4096)), dim3(256), 0, st, pa_fused, a);
  } else {
    launch_score<D, K_SAMPLE>(make_score_args(p, K_SAMPLE), p.head_mode, 4096, st);
  }
  if (p.hm_prob) {
    hipLaunchKernelGGL(k_lhat, dim3(lists * p.Hq), dim3(1024), 0, st, la);
    hipLaunchKernelGGL(k_alpha, dim3(lists, cdiv(p.m_max, 256)), dim3(256), 0, st, la, p.alpha);
    ListArgs lt = la;   // the cut-off over the estimated attention of the sample
    lt.samp = p.alpha;
    launch_thresh(lt, lists, p.m_max, false, st);
  } else if (!pt) {
    launch_thresh(la, lists, p.m_max, lists > 2 * cus, st);
  }
  // 4. streaming pass over every key row
  if (p.ev_start) (void)hipEventRecord(p.ev_start, st);
  if (p.head_mode == 0) {
    ScoreArgs a = make_score_args(p, K_STREAM);
    a.score_mode = p.score_mode;
    a.below = p.below;
    const int64_t tiles = a.tile_base[p.S];
    if (tiles > 0) {
      const int grid = (int)std::min<int64_t>(stream_grid<D, 0>(), std::max<int64_t>(1, tiles / 16));
      int nseg = 0;   // (stream, layer, KV head) segments with rows
      for (int s = 0; s < p.S; ++s) nseg += a.ntile[s] > 0 ? p.L * p.Hk : 0;
      a.sgroup = stream_group(grid, nseg);
      a.xcd_weights = cus == 256;
      if (a.sgroup < kStreamGroupMax) a.dyn_tiles = tiles * kDynPermille / 1000;
      hipLaunchKernelGGL(k_stream<D>, dim3(grid), dim3(256), 0, st, a);
    }
  } else {
    ScoreArgs a = make_score_args(p, K_STREAM);
    int64_t tiles = 0;   // segments are (stream, layer)
    for (int s = 0; s < p.S; ++s) {
      a.tile_base[s] = tiles;
      tiles += (int64_t)p.L * a.ntile[s];
    }
    a.tile_base[p.S] = tiles;
    if (tiles > 0 && p.hm_prob) {
      a.score_mode = 1;
      a.below = p.below;
      a.lhat = p.lhat;
      a.left_max = p.left_max;
      const hipError_t e = launch_stream_hp<D>(a, p, tiles, cus, st);
      if (e != hipSuccess) return e;
    } else if (tiles > 0) {
      const int grid = (int)std::min<int64_t>(stream_grid<D, 1>(), std::max<int64_t>(1, tiles / 16));
      int nseg = 0;   // (stream, layer) segments with rows
      for (int s = 0; s < p.S; ++s) nseg += a.ntile[s] > 0 ? p.L : 0;
      a.sgroup = stream_group(grid, nseg);
      a.xcd_weights = cus == 256;
      hipLaunchKernelGGL(k_stream_hm<D>, dim3(grid), dim3(256), 0, st, a);
    }
  }
  if (p.ev_stop) (void)hipEventRecord(p.ev_stop, st);
  // 5. exact top-k from candidates (6. exact fallback for flagged lists), each
  // list adding its votes and mass per frame; 7. the pool
  VoteArgs va{};
  va.NL = p.NL; va.k_max = p.k_max; va.pool = p.pool; va.f_max = p.f_max;
  va.hist_stride = p.dbg_hist_stride;
  for (int s = 0; s < p.S; ++s) {
    va.f[s] = p.st[s].f;
    va.frame0[s] = p.st[s].frame0;
    va.hist0[s] = p.st[s].hist0;
  }
  va.votes_g = p.votes; va.massfx_g = p.massfx; va.sexp = p.sexp;
  va.rec_hi = p.rec_hi; va.rec_lo = p.rec_lo;
  va.pool_ids = p.pool_ids; va.pool_votes = p.pool_votes; va.pool_mass = p.pool_mass;
  va.pool_n = p.pool_n;
  va.dbg_vote_hist = p.dbg_vote_hist; va.dbg_mass_hist = p.dbg_mass_hist;
  va.dbg_pool = p.dbg_pool; va.dbg_pool_n = p.dbg_pool_n;
  if (p.hm_prob) {
    const dim3 cg(lists, cdiv(p.cap, 64));
    switch (p.Hk) {   // the streaming pass's KV-head counts
      case 1: hipLaunchKernelGGL((k_cand_logits<D, 1>), cg, dim3(256), 0, st, la); break;
      case 2: hipLaunchKernelGGL((k_cand_logits<D, 2>), cg, dim3(256), 0, st, la); break;
      case 4: hipLaunchKernelGGL((k_cand_logits<D, 4>), cg, dim3(256), 0, st, la); break;
      case 8:   // as the streaming pass: H_kv = 8 only at head dimension 64
        if (D * 8 <= 512) hipLaunchKernelGGL((k_cand_logits<D, (D * 8 <= 512 ? 8 : 4)>), cg, dim3(256), 0, st, la);
        break;
      default: break;
    }
    hipLaunchKernelGGL(k_cand_lse, dim3(lists * p.Hq), dim3(256), 0, st, la);
    hipLaunchKernelGGL(k_select_hp<D>, dim3(lists), dim3(1024), 0, st, la);
  }
  else if (lists > 2 * cus) hipLaunchKernelGGL(k_select_dense<D>, dim3(lists), dim3(1024), 0, st, la);
  else hipLaunchKernelGGL(k_select<D>, dim3(lists), dim3(1024), 0, st, la);
  // 8. Gram matrix, 9. max-min
  GramArgs ga{};
  ga.pool = p.pool; ga.ld = (p.pool + 3) & ~3; ga.dim = p.Hk * D; ga.tiles = cdiv(p.pool, 16);
  for (int s = 0; s < p.S; ++s) ga.desc[s] = p.st[s].desc;
  ga.pool_ids = p.pool_ids; ga.pool_n = p.pool_n; ga.gram = p.gram;
  MaxminArgs ma{};
  ma.pool = p.pool; ma.ld = ga.ld; ma.n_select = p.n_select;
  ma.pool_ids = p.pool_ids; ma.pool_votes = p.pool_votes; ma.pool_mass = p.pool_mass;
  ma.pool_n = p.pool_n; ma.gram = p.gram;
  for (int s = 0; s < p.S; ++s) ma.frame0[s] = p.st[s].frame0;
  ma.out_ids = p.out_ids; ma.out_votes = p.out_votes; ma.out_mass = p.out_mass; ma.out_n = p.out_n;
  if (ga.dim % 64 != 0 || ga.dim < 64 || ga.dim > kMaxDescDim) return hipErrorInvalidValue;
  // pool and Gram matrix in one launch when every record fits in LDS
  const bool pool_gram = p.f_max <= kPoolSort;
  if (!pool_gram) hipLaunchKernelGGL(k_votes_pool, dim3(p.S), dim3(1024), 0, st, va);
  gram_launchers<kMaxDescDim / 64>()[ga.dim / 64 - 1](dim3(p.S * ga.tiles * ga.tiles), pool_gram ? &va : nullptr,
                                                      ga, st);
  hipLaunchKernelGGL(k_maxmin, dim3(p.S), dim3(1024), 0, st, ma);
  return hipGetLastError();
}

template <int D>
hipError_t debug_scores_impl(RetrievePlan& p, int layer, int q_head, int64_t row0, int64_t n_rows,
                             float* out, hipStream_t st) {
  PrepArgs pa{};
  pa.Hq = p.Hq; pa.Hk = p.Hk; pa.G = p.G; pa.L = p.L; pa.head_mode = p.head_mode; pa.first = 0;
  for (int l = 0; l < p.L; ++l) pa.q[l] = p.st[0].q[l];
  pa.nq[0] = p.st[0].nq; pa.qscale[0] = p.st[0].qscale;
  pa.qB = reinterpret_cast<u32x4*>(p.qB);
  hipLaunchKernelGGL(k_prep<D>, dim3(p.L * p.Hk), dim3(8 * D), 0, st, pa);
  ScoreArgs a{};
  a.L = p.L; a.Hq = p.Hq; a.Hk = p.Hk; a.G = p.G; a.NL = p.NL; a.ngs = p.ngs;
  a.head_mode = p.head_mode; a.S = 1; a.chunk = p.chunk_rows;
  a.qB = reinterpret_cast<const u32x4*>(p.qB);
  a.keys[0] = p.st[0].keys; a.stride[0] = p.st[0].row_stride; a.n[0] = (int32_t)n_rows;
  a.units[0] = (int32_t)n_rows;
  // only the item range of the requested (layer, KV head) is enumerated
  const int nch = cdiv(n_rows, a.chunk);
  a.item_base[0] = 0;
  a.item_base[1] = p.L * p.ngs * nch;
  a.total_items = a.item_base[1];
  a.only_list = p.head_mode == 0 ? layer * p.Hq + q_head : layer;
  a.full = out; a.full_base[0] = -(int64_t)a.only_list * n_rows; a.full_stride[0] = (int32_t)n_rows;
  a.row0 = row0;
  if (n_rows > 0) launch_score<D, K_FULL>(a, p.head_mode, 2048, st);
  return hipGetLastError();
}

}  // namespace

size_t pooled_workspace(PooledPlan& p, void* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    off = (off + 255) & ~(size_t)255;
    void* r = ws ? static_cast<char*>(ws) + off : nullptr;
    off += bytes;
    return r;
  };
  p.w = static_cast<float*>(take((size_t)p.S * p.L * p.Hk * p.D * 4));
  p.scores = static_cast<float*>(take((size_t)p.S * std::max<int64_t>(p.f_max, 1) * 4));
  return (off + 255) & ~(size_t)255;
}

template <int D>
hipError_t pooled_impl(const PooledPlan& p, hipStream_t st) {
  const int pairs = p.S * p.L;
  for (int first = 0; first < pairs; first += 128) {
    PoolQArgs a{};
    a.Hq = p.Hq; a.Hk = p.Hk; a.G = p.G; a.L = p.L; a.first = first; a.w = p.w;
    const int cnt = std::min(128, pairs - first);
    for (int i = 0; i < cnt; ++i) a.q[i] = p.q[first + i];
    for (int s = 0; s < p.S; ++s) a.nq[s] = p.nq[s];
    hipLaunchKernelGGL(k_pool_query<D>, dim3(cnt * p.Hk), dim3(kPoolQGroups * D), 0, st, a);
  }
  PoolScoreArgs sa{};
  sa.n4 = p.L * p.Hk * D / 4;
  sa.w = reinterpret_cast<const float4*>(p.w);
  sa.scores = p.scores;
  sa.f_max = std::max<int64_t>(p.f_max, 1);
  PoolSelectArgs ka{};
  ka.n_select = p.n_select; ka.scores = p.scores; ka.f_max = sa.f_max;
  ka.out_ids = p.out_ids; ka.out_scores = p.out_scores; ka.out_n = p.out_n;
  for (int s = 0; s < p.S; ++s) {
    sa.F[s] = p.F[s];
    sa.pooled[s] = reinterpret_cast<const float4*>(p.pooled[s]);
    ka.F[s] = p.F[s];
    ka.frame0[s] = p.frame0[s];
  }
  if (p.f_max > 0)
    hipLaunchKernelGGL(k_pool_score, dim3((unsigned)cdiv(p.f_max, 4), p.S), dim3(256), 0, st, sa);
  hipLaunchKernelGGL(k_pool_select, dim3(p.S), dim3(1024), 0, st, ka);
  return hipGetLastError();
}

hipError_t launch_pooled(const PooledPlan& p, hipStream_t st) {
  return p.D == 64 ? pooled_impl<64>(p, st) : pooled_impl<128>(p, st);
}

hipError_t launch_zero32(int32_t* p, int n, hipStream_t st) {
  hipLaunchKernelGGL(k_zero32, dim3(1), dim3(64), 0, st, p, n);
  return hipGetLastError();
}

hipError_t launch_absorb(const AbsorbArgs& a, hipStream_t st) {
  if (a.n_units <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_cluster_assign, dim3(1), dim3(256), 0, st, a);
  const int64_t E = (int64_t)a.L * a.Hk * a.R * a.D;
  hipLaunchKernelGGL(k_cluster_reps, dim3((unsigned)cdiv(E, 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

size_t cluster_query_workspace(ClusterQueryPlan& p, void* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    off = (off + 255) & ~(size_t)255;
    void* r = ws ? static_cast<char*>(ws) + off : nullptr;
    off += bytes;
    return r;
  };
  p.w = static_cast<float*>(take((size_t)p.Hk * p.D * 4));
  p.scores = static_cast<float*>(take((size_t)std::max<int64_t>(p.max_clusters, 1) * 4));
  return (off + 255) & ~(size_t)255;
}

template <int D>
hipError_t cluster_query_impl(const ClusterQueryPlan& p, hipStream_t st) {
  // the last layer's pooled query weights (one layer: scale 1/(n_q H_q sqrt d))
  PoolQArgs qa{};
  qa.Hq = p.Hq; qa.Hk = p.Hk; qa.G = p.G; qa.L = 1; qa.first = 0; qa.w = p.w;
  qa.q[0] = p.q_last;
  qa.nq[0] = p.nq;
  hipLaunchKernelGGL(k_pool_query<D>, dim3(p.Hk), dim3(kPoolQGroups * D), 0, st, qa);
  PoolScoreArgs sa{};
  sa.n4 = p.Hk * D / 4;
  sa.count = p.cl.state;
  sa.F[0] = p.max_clusters;
  sa.pooled[0] = reinterpret_cast<const float4*>(p.cl.centroids);
  sa.w = reinterpret_cast<const float4*>(p.w);
  sa.scores = p.scores;
  sa.f_max = std::max<int64_t>(p.max_clusters, 1);
  hipLaunchKernelGGL(k_pool_score, dim3((unsigned)cdiv(p.max_clusters, 4), 1), dim3(256), 0, st, sa);
  PoolSelectArgs ka{};
  ka.n_select = p.k;
  ka.count = p.cl.state;
  ka.span = p.cl.span;
  ka.out_first = p.out_first;
  ka.out_last = p.out_last;
  ka.F[0] = p.max_clusters;
  ka.frame0[0] = 0;
  ka.scores = p.scores;
  ka.f_max = sa.f_max;
  ka.out_ids = p.out_ids;
  ka.out_scores = p.out_scores;
  ka.out_n = p.out_n;
  hipLaunchKernelGGL(k_pool_select, dim3(1), dim3(1024), 0, st, ka);
  return hipGetLastError();
}

hipError_t launch_cluster_query(const ClusterQueryPlan& p, hipStream_t st) {
  return p.D == 64 ? cluster_query_impl<64>(p, st) : cluster_query_impl<128>(p, st);
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t st) {
  auto grid = [](int64_t n) { return dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192))); };
  // items [shift, shift + keep) -> [0, keep) of `unit` units each, in passes of at most `shift` items
  auto move16 = [&](void* base, int64_t seg_stride, int n_seg, int64_t unit, int64_t shift, int64_t keep) {
    for (int64_t done = 0; done < keep; done += shift) {
      const int64_t len = std::min(shift, keep - done) * unit;
      hipLaunchKernelGGL(k_move16, grid(len * n_seg), dim3(256), 0, st, static_cast<u32x4*>(base), seg_stride,
                         n_seg, (shift + done) * unit, done * unit, len);
    }
  };
  auto move4 = [&](void* base, int64_t seg_stride, int n_seg, int64_t shift, int64_t keep, uint32_t sub) {
    for (int64_t done = 0; done < keep; done += shift) {
      const int64_t len = std::min(shift, keep - done);
      hipLaunchKernelGGL(k_move4, grid(len * n_seg), dim3(256), 0, st, static_cast<uint32_t*>(base), seg_stride,
                         n_seg, shift + done, done, len, sub);
    }
  };
  const int lg = a.L * a.Hk;
  if (a.row_shift > 0 && a.keep_rows > 0) {
    move16(a.dev.keys, a.max_rows * a.D / 8, lg, a.D / 8, a.row_shift, a.keep_rows);   // 16-byte units of bf16 rows
    move4(a.dev.counts, a.max_rows, lg, a.row_shift, a.keep_rows, 0u);
  }
  if (a.frame_shift > 0) {
    if (a.keep_frames > 0) {
      move16(a.dev.desc, 0, 1, (int64_t)a.Hk * a.D / 4, a.frame_shift, a.keep_frames);
      move16(a.dev.pooled, 0, 1, (int64_t)a.L * a.Hk * a.D / 4, a.frame_shift, a.keep_frames);
    }
    move4(a.dev.frame_off, 0, 1, a.frame_shift, a.keep_frames + 1, (uint32_t)a.row_shift);
  }
  return hipGetLastError();
}

hipError_t launch_evidence(const EvidenceArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_evidence, dim3(a.S), dim3(256), 0, st, a);
  return hipGetLastError();
}

size_t carve_workspace(RetrievePlan& p, void* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    off = (off + 255) & ~(size_t)255;
    void* r = ws ? static_cast<char*>(ws) + off : nullptr;
    off += bytes;
    return r;
  };
  const size_t lists = (size_t)p.S * p.NL;
  p.qB = static_cast<uint32_t*>(take((size_t)p.S * p.L * p.Hk * 2 * (p.D / 32) * 64 * 16));
  p.tau = static_cast<uint32_t*>(take(lists * 4));
  p.cnt = static_cast<uint32_t*>(take(lists * 4));
  p.samp = static_cast<float*>(take((size_t)p.S * p.NLs * (size_t)p.m_max * 4));
  p.below = p.score_mode == 1 ? static_cast<uint64_t*>(take((size_t)p.S * p.NLs * 8)) : nullptr;
  p.lhat = p.hm_prob ? static_cast<float*>(take((size_t)p.S * p.NLs * 4)) : nullptr;
  p.cand_sc = p.hm_prob ? static_cast<float*>(take(lists * (size_t)p.cap * p.Hq * 4)) : nullptr;
  p.left_max = p.hm_prob ? static_cast<uint32_t*>(take(lists * 4)) : nullptr;
  p.alpha = p.hm_prob ? static_cast<float*>(take(lists * (size_t)p.m_max * 4)) : nullptr;
  p.cand_lse = p.hm_prob ? static_cast<float*>(take(lists * (size_t)p.Hq * 4)) : nullptr;
  p.cand = static_cast<uint64_t*>(take(lists * (size_t)p.cap * 8));
  p.qcol = static_cast<float*>(take((size_t)p.S * p.L * p.Hk * 16 * 4));
  p.sexp = static_cast<int32_t*>(take((size_t)p.S * 4));
  p.dyn_ctr = static_cast<uint32_t*>(take((size_t)kDynCtr * kDynStride * 4));
  p.votes = static_cast<int32_t*>(take((size_t)p.S * p.f_max * 4));
  p.massfx = static_cast<int64_t*>(take((size_t)p.S * p.f_max * 8));
  p.rec_hi = static_cast<uint64_t*>(take((size_t)p.S * p.f_max * 8));
  p.rec_lo = static_cast<uint64_t*>(take((size_t)p.S * p.f_max * 8));
  p.pool_ids = static_cast<int32_t*>(take((size_t)p.S * p.pool * 4));
  p.pool_votes = static_cast<int32_t*>(take((size_t)p.S * p.pool * 4));
  p.pool_mass = static_cast<float*>(take((size_t)p.S * p.pool * 4));
  p.pool_n = static_cast<int32_t*>(take((size_t)p.S * 4));
  p.gram = static_cast<float*>(take((size_t)p.S * p.pool * ((p.pool + 3) & ~3) * 4));
  return (off + 255) & ~(size_t)255;
}

hipError_t launch_append(const AppendArgs& a, bool compress, hipStream_t st) {
  return a.D == 128 ? append_impl<128>(a, compress, st) : append_impl<64>(a, compress, st);
}

// The no-alloc retrieval's workspace.  In host code `scratch` names a host-side
// stand-in, not device memory: only the address that hipGetSymbolAddress
// returns for the current device is ever passed to a kernel.  The runtime
// places one copy on each device when the library's code object is loaded
// there; it lives until the process ends.
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

hipError_t noalloc_workspace(void** ptr) {
  static std::atomic<void*> cache[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = cache[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    // concurrent first calls on one device look up the same address
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    cache[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return hipSuccess;
}

hipError_t launch_retrieve(RetrievePlan& p, hipStream_t st) {
  return p.D == 128 ? retrieve_impl<128>(p, st) : retrieve_impl<64>(p, st);
}

hipError_t launch_debug_scores(RetrievePlan& p, int layer, int q_head, int64_t row0,
                               int64_t n_rows, float* out, hipStream_t st) {
  return p.D == 128 ? debug_scores_impl<128>(p, layer, q_head, row0, n_rows, out, st)
                    : debug_scores_impl<64>(p, layer, q_head, row0, n_rows, out, st);
}

}  // namespace ss
