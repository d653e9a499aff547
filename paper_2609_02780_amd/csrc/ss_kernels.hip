// gfx950 (MI355X) kernels for ShallowStream's query-time evidence retrieval.
//
// Retrieval pipeline (Sec. 4.2 "Optional Evidence Retrieval"), all on one HIP
// stream, no host synchronisation:
//   k_prep      mean query per (layer, head), pre-scaled, split into bf16 hi+lo
//               and laid out as the MFMA B operand (lane-native).
//   k_score<SAMPLE>   scores of a strided sample of rows per list.
//   k_thresh    per list, the r-th largest sample score: a cut-off that keeps at
//               least r >= ... rows of the full list (see the host planner).
//   k_score<STREAM>   THE HOT KERNEL: streams every bf16 key row from HBM once,
//               bf16 MFMA (16x16x32) against the group's query columns with fp32
//               accumulation, appends rows scoring >= the cut-off as 64-bit
//               composite keys (ordered score, inverted row).
//   k_select    exact top-k per list from the candidates (radix select + bitonic
//               sort in LDS); lists whose candidate count fell outside
//               [k, capacity] are flagged.
//   k_score<FULL> + k_fb_select   exact fallback for flagged lists only:
//               materialise every score, radix select, ties by row order.
//   k_votes_pool  one vote per selected row for its frame, attention mass in
//               deterministic fixed point, vote-ranked pool (bitonic in LDS).
//   k_gram      pool descriptor Gram matrix (fp32).
//   k_maxmin    greedy max-min diversity over the Gram matrix.
//
// Append: k_desc (Eq. memory_key descriptor), k_copy (raw rows) or k_kmeans
// (per-frame k-means compression).
//
// Ordering conventions: a score s maps to an order-preserving uint32 u(s); the
// composite key (u(s) << 32) | (0xFFFFFFFF - row) sorts descending exactly as
// (score desc, row asc), the top-k tie rule.
#include "ss_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>

namespace ss {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kSelLds = 8192;       // candidates staged in LDS by k_select
constexpr int kVoteLds = 4096;      // frames whose votes/mass live in LDS
constexpr int kPoolSort = 4096;     // records per pool sorting round

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

__device__ __forceinline__ u32x4 ld_nt(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Exclusive prefix count of `p` among the lanes of a wave.
__device__ __forceinline__ int wave_excl_count(bool p) {
  const uint64_t m = __ballot(p);
  const int lane = threadIdx.x & (kWave - 1);
  return __popcll(m & ((1ull << lane) - 1ull));
}

// Block-wide exclusive scan of `v`; `sh` needs blockDim/64 + 1 ints.  Returns the
// thread's exclusive prefix; `total` receives the block sum.
__device__ int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
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
    uint32_t x = mine;  // inclusive suffix sum over lanes >= lane
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t y = __shfl_down(x, o);
      if (lane + o < kWave) x += y;
    }
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
};

// One wave per (stream, layer, KV head).  Lane (col = lane % 16, kg = lane / 16)
// owns column col of the B tile and, at k-step i, the 8 dims 32 i + 8 kg .. +7.
// Column c of head-mode 0 is query head g*G + c; head-mode 1 uses column 0 only,
// holding the sum of the group's head means (the layer's head average is the
// sum over KV heads of these columns against their keys).
template <int D>
__global__ __launch_bounds__(64) void k_prep(PrepArgs a) {
  constexpr int KS = D / 32;
  const int pair_local = blockIdx.x / a.Hk, g = blockIdx.x % a.Hk;
  const int pair = a.first + pair_local;
  const int s = pair / a.L;
  const uint16_t* q = a.q[pair_local];
  const int nq = a.nq[s];
  const float scale = a.qscale[s];
  const int lane = threadIdx.x, col = lane & 15, kg = lane >> 4;
  int h0, h1;
  if (a.head_mode == 0) {
    h0 = g * a.G + col;
    h1 = (col < a.G) ? h0 + 1 : h0;
  } else {
    h0 = g * a.G;
    h1 = (col == 0) ? h0 + a.G : h0;
  }
  u32x4* out = a.qB + ((size_t)pair * a.Hk + g) * (2 * KS * kWave);
  for (int i = 0; i < KS; ++i) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int e0 = 32 * i + 8 * kg;
    for (int h = h0; h < h1; ++h) {
      for (int j = 0; j < nq; ++j) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(q + ((size_t)h * nq + j) * D + e0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          acc[2 * t] += bf16_lo(v[t]);
          acc[2 * t + 1] += bf16_hi(v[t]);
        }
      }
    }
    u32x4 hi, lo;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float x0 = acc[2 * t] * scale, x1 = acc[2 * t + 1] * scale;
      const uint16_t a0 = bf16_rne(x0), a1 = bf16_rne(x1);
      const uint16_t b0 = bf16_rne(x0 - __uint_as_float((uint32_t)a0 << 16));
      const uint16_t b1 = bf16_rne(x1 - __uint_as_float((uint32_t)a1 << 16));
      hi[t] = (uint32_t)a0 | ((uint32_t)a1 << 16);
      lo[t] = (uint32_t)b0 | ((uint32_t)b1 << 16);
    }
    out[(0 * KS + i) * kWave + lane] = hi;
    out[(1 * KS + i) * kWave + lane] = lo;
  }
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
  // K_STREAM
  const uint32_t* tau;
  uint32_t* cnt;
  uint64_t* cand;
  int cap;
  // K_FULL
  const int32_t* flag;                // nullptr: write only `only_list`
  int only_list;
  float* full;
  int64_t full_base[kMaxStreams];
  int32_t full_stride[kMaxStreams];
  int64_t row0;
};

// Row of the key index scored for unit u of stream s.
template <int KIND>
__device__ __forceinline__ int64_t unit_row(const ScoreArgs& a, int s, int u) {
  if (KIND == K_SAMPLE) {
    // evenly spread sample: row floor((2u+1) n / (2m)), the identity when m == n
    const int64_t n = a.n[s], m = a.units[s];
    return ((2 * (int64_t)u + 1) * n) / (2 * m);
  } else if (KIND == K_FULL) {
    return a.row0 + u;
  } else {
    return u;
  }
}

// Per-lane output of one 16-row tile: lane (col, kg) holds the scores of rows
// 4 kg + j (j < 4) of the tile for output column col.
template <int KIND>
__device__ __forceinline__ void emit(const ScoreArgs& a, int s, int list, bool colv, bool wr,
                                     uint32_t tau_u, int tile_u0, int u1, f32x4 acc, int kg,
                                     bool& ovf) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int u = tile_u0 + 4 * kg + j;
    const float sc = acc[j] + 0.0f;  // canonical zero: -0 becomes +0
    if (KIND == K_SAMPLE) {
      if (colv && u < u1) a.samp[(size_t)list * a.samp_stride + u] = sc;
    } else if (KIND == K_STREAM) {
      const uint32_t uo = ord_u32(sc);
      if (colv && u < u1 && uo >= tau_u && !ovf) {
        const uint32_t slot = atomicAdd(&a.cnt[list], 1u);
        if (slot < (uint32_t)a.cap) {
          a.cand[(size_t)list * a.cap + slot] = mk_key(uo, (uint32_t)u);
        } else {
          ovf = true;  // the list will take the exact fallback; stop counting
        }
      }
    } else {
      if (wr && u < u1) {
        const int ll = list - s * a.NL;
        a.full[a.full_base[s] + (int64_t)ll * a.full_stride[s] + u] = sc;
      }
    }
  }
}

// Head-mode 0: one KV head per item, its G query heads in the MFMA columns, the
// B operand in registers, two tiles in flight per wave.
template <int D, int KIND>
__global__ __launch_bounds__(256) void k_score(ScoreArgs a) {
  constexpr int KS = D / 32;
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
      wr = colv && (a.flag ? (a.flag[list] != 0) : (ll == a.only_list));
      if (!__any(wr)) continue;  // same decision in every wave of the block
    }
    uint32_t tau_u = 0xFFFFFFFFu;
    if (KIND == K_STREAM && colv) tau_u = a.tau[list];
    bool ovf = false;
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
    auto compute = [&](int t, const u32x4 (&A)[KS]) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < KS; ++i) {
        acc = mfma_bf16(A[i], bh[i], acc);
        acc = mfma_bf16(A[i], bl[i], acc);
      }
      emit<KIND>(a, s, list, colv, wr, tau_u, u0 + t * kTile, u1, acc, kg, ovf);
    };

    u32x4 A0[KS], A1[KS];
    int t = wave;
    load(t, A0);
    for (; t < ntiles; t += 2 * nw) {
      load(t + nw, A1);
      compute(t, A0);
      if (t + nw >= ntiles) break;
      load(t + 2 * nw, A0);
      compute(t + nw, A1);
    }
  }
}

// Head-mode 1: every KV head of the layer accumulates into column 0 (the
// layer's head-averaged score); B tiles of all KV heads staged in LDS.
template <int D, int KIND>
__global__ __launch_bounds__(256) void k_score_hm(ScoreArgs a) {
  constexpr int KS = D / 32;
  __shared__ u32x4 sB[8 * 2 * KS * kWave];  // H_kv <= 8 in head-mode 1
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int col = lane & 15, kg = lane >> 4, rl = lane & 15;
  for (int item = blockIdx.x; item < a.total_items; item += gridDim.x) {
    int s = 0;
    while (item >= a.item_base[s + 1]) ++s;
    const int rem = item - a.item_base[s];
    const int units = a.units[s];
    const int nch = (units + a.chunk - 1) / a.chunk;
    const int chunk = rem % nch, l = rem / nch;
    const int u0 = chunk * a.chunk, u1 = min(units, u0 + a.chunk);
    const bool colv = col == 0;
    const int list = s * a.NL + l;
    bool wr = false;
    if (KIND == K_FULL) {
      wr = colv && (a.flag ? (a.flag[list] != 0) : (l == a.only_list));
      if (!__any(wr)) continue;
    }
    uint32_t tau_u = 0xFFFFFFFFu;
    if (KIND == K_STREAM && colv) tau_u = a.tau[list];
    bool ovf = false;
    __syncthreads();
    const u32x4* qb = a.qB + (size_t)(s * a.L + l) * a.Hk * (2 * KS * kWave);
    for (int i = threadIdx.x; i < a.Hk * 2 * KS * kWave; i += blockDim.x) sB[i] = qb[i];
    __syncthreads();
    const size_t gstride = (size_t)a.stride[s] * D;
    const uint16_t* base = a.keys[s] + (size_t)l * a.Hk * gstride + 8 * kg;
    const int ntiles = (u1 - u0 + kTile - 1) / kTile;
    for (int t = wave; t < ntiles; t += nw) {
      const int u = u0 + t * kTile + rl;
      const bool ok = u < u1;
      const int64_t row = ok ? unit_row<KIND>(a, s, u) : 0;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int g = 0; g < a.Hk; ++g) {
        const uint16_t* p = base + g * gstride + row * D;
        u32x4 A[KS];
#pragma unroll
        for (int i = 0; i < KS; ++i) A[i] = ok ? ld_nt(p + 32 * i) : u32x4{0, 0, 0, 0};
        const u32x4* b = sB + g * (2 * KS * kWave);
#pragma unroll
        for (int i = 0; i < KS; ++i) {
          acc = mfma_bf16(A[i], b[i * kWave + lane], acc);
          acc = mfma_bf16(A[i], b[(KS + i) * kWave + lane], acc);
        }
      }
      emit<KIND>(a, s, list, colv, wr, tau_u, u0 + t * kTile, u1, acc, kg, ovf);
    }
  }
}

// ---------------------------------------------------------------------------
// k_thresh: per list, the r-th largest sample score as an ordered uint32
// ---------------------------------------------------------------------------
struct ListArgs {
  int NL, S, cap, k_max, top_k;
  int32_t m[kMaxStreams], r[kMaxStreams], kk[kMaxStreams], n[kMaxStreams];
  int64_t full_base[kMaxStreams];
  const float* samp;
  int samp_stride;
  uint32_t* tau;
  uint32_t* cnt;
  int32_t* flag;
  const uint64_t* cand;
  uint64_t* topk;
  const float* full;
  int32_t* dbg_pos;
  float* dbg_score;
  int32_t* dbg_stats;
};

__global__ __launch_bounds__(256) void k_thresh(ListArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t res[4];
  const int list = blockIdx.x, s = list / a.NL;
  const int m = a.m[s], r = a.r[s];
  if (threadIdx.x == 0) {
    a.cnt[list] = 0;
    a.flag[list] = 0;
  }
  if (m == 0 || r == 0) {
    if (threadIdx.x == 0) a.tau[list] = 0xFFFFFFFFu;
    return;
  }
  const float* v = a.samp + (size_t)list * a.samp_stride;
  uint32_t ngt;
  const uint32_t t = radix_select_u32([&](int i) { return ord_u32(v[i]); }, m, (uint32_t)r, hist,
                                      res, ngt);
  if (threadIdx.x == 0) a.tau[list] = t;
}

// ---------------------------------------------------------------------------
// k_select: exact top-k of a list's candidates
// ---------------------------------------------------------------------------
__device__ void write_topk(const ListArgs& a, int list, const uint64_t* sorted, int kk) {
  uint64_t* out = a.topk + (size_t)list * a.k_max;
  for (int i = threadIdx.x; i < kk; i += blockDim.x) out[i] = sorted[i];
  if (a.dbg_pos) {
    int32_t* dp = a.dbg_pos + (size_t)list * a.top_k;
    float* ds = a.dbg_score + (size_t)list * a.top_k;
    for (int i = threadIdx.x; i < a.top_k; i += blockDim.x) {
      dp[i] = i < kk ? (int32_t)key_row(sorted[i]) : -1;
      ds[i] = i < kk ? key_score(sorted[i]) : 0.f;
    }
  }
}

__global__ __launch_bounds__(256) void k_select(ListArgs a) {
  __shared__ uint64_t stage[kSelLds];
  __shared__ uint64_t sorted[kMaxTopK];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t res[4];
  __shared__ uint32_t ngather;
  const int list = blockIdx.x, s = list / a.NL;
  const int kk = a.kk[s];
  if (kk == 0) {
    write_topk(a, list, sorted, 0);
    return;
  }
  const uint32_t c = a.cnt[list];
  if (c < (uint32_t)kk || c > (uint32_t)a.cap) {
    if (threadIdx.x == 0) a.flag[list] = 1;
    return;
  }
  const int n = (int)c;
  const uint64_t* src = a.cand + (size_t)list * a.cap;
  const bool in_lds = n <= kSelLds;
  if (in_lds) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) stage[i] = src[i];
    __syncthreads();
  }
  const uint64_t* v = in_lds ? stage : src;
  const uint64_t cut = radix_select_u64([&](int i) { return v[i]; }, n, (uint32_t)kk, hist, res);
  if (threadIdx.x == 0) ngather = 0;
  const int np = pow2_ceil(kk);
  for (int i = kk + threadIdx.x; i < np; i += blockDim.x) sorted[i] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const uint64_t x = v[i];
    if (x >= cut) {
      const uint32_t slot = atomicAdd(&ngather, 1u);
      if (slot < (uint32_t)np) sorted[slot] = x;
    }
  }
  __syncthreads();
  bitonic_desc_u64(sorted, np);
  write_topk(a, list, sorted, kk);
}

// Exact fallback: every score of the list was materialised by k_score<FULL>.
__global__ __launch_bounds__(256) void k_fb_select(ListArgs a) {
  __shared__ uint64_t sorted[kMaxTopK];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t res[4];
  __shared__ uint32_t ngt_sh;
  __shared__ int scan_sh[8];
  const int list = blockIdx.x, s = list / a.NL;
  if (a.dbg_stats && threadIdx.x == 0) {
    a.dbg_stats[2 * list] = (int32_t)min(a.cnt[list], (uint32_t)INT_MAX);
    a.dbg_stats[2 * list + 1] = a.flag[list];
  }
  if (!a.flag[list]) return;
  const int kk = a.kk[s], n = a.n[s];
  const float* v = a.full + a.full_base[s] + (int64_t)(list - s * a.NL) * n;
  uint32_t ngreater;
  const uint32_t vstar = radix_select_u32([&](int i) { return ord_u32(v[i]); }, n,
                                          (uint32_t)kk, hist, res, ngreater);
  const int need_eq = kk - (int)ngreater;
  const int np = pow2_ceil(kk);
  if (threadIdx.x == 0) ngt_sh = 0;
  for (int i = kk + threadIdx.x; i < np; i += blockDim.x) sorted[i] = 0;
  __syncthreads();
  // rows scoring above v* in any order; rows equal to v* in row order until need_eq
  int eq_taken = 0;
  for (int b0 = 0; b0 < n; b0 += blockDim.x) {
    const int i = b0 + threadIdx.x;
    uint32_t u = 0;
    bool gt = false, eq = false;
    if (i < n) {
      u = ord_u32(v[i]);
      gt = u > vstar;
      eq = u == vstar;
    }
    if (gt) {
      const uint32_t slot = atomicAdd(&ngt_sh, 1u);
      if (slot < (uint32_t)np) sorted[slot] = mk_key(u, (uint32_t)i);
    }
    int tot;
    const int pre = block_excl_scan(eq ? 1 : 0, scan_sh, tot);
    if (eq && eq_taken + pre < need_eq) sorted[ngreater + eq_taken + pre] = mk_key(u, (uint32_t)i);
    eq_taken += tot;
  }
  __syncthreads();
  bitonic_desc_u64(sorted, np);
  write_topk(a, list, sorted, kk);
}

// ---------------------------------------------------------------------------
// k_votes_pool: votes, attention mass and the vote-ranked pool (one block per stream)
// ---------------------------------------------------------------------------
struct VoteArgs {
  int NL, k_max, pool, f_max, hist_stride;
  int32_t kk[kMaxStreams], f[kMaxStreams], rpf[kMaxStreams];
  const int32_t* frame_off[kMaxStreams];
  const uint64_t* topk;
  int32_t* votes_g;     // [S][f_max] (frames beyond the LDS capacity)
  int64_t* massfx_g;    // [S][f_max]
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

__device__ __forceinline__ int frame_of(const VoteArgs& a, int s, uint32_t row) {
  if (a.rpf[s] > 0) return (int)(row / (uint32_t)a.rpf[s]);
  const int32_t* off = a.frame_off[s];
  int lo = 0, hi = a.f[s] - 1;  // largest f with off[f] <= row
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((uint32_t)off[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(1024) void k_votes_pool(VoteArgs a) {
  __shared__ int32_t sv[kVoteLds];
  __shared__ int64_t sm[kVoteLds];
  __shared__ uint64_t shi[kPoolSort];
  __shared__ uint64_t slo[kPoolSort];
  __shared__ float red[16];
  __shared__ int scan_sh[17];
  const int s = blockIdx.x;
  const int kk = a.kk[s], F = a.f[s], NL = a.NL;
  const int E = NL * kk;
  const uint64_t* tk = a.topk + (size_t)s * NL * a.k_max;
  const bool lds = F <= kVoteLds;
  int32_t* votes = lds ? sv : a.votes_g + (size_t)s * a.f_max;
  int64_t* massfx = lds ? sm : a.massfx_g + (size_t)s * a.f_max;

  // fixed-point exponent: |sum| <= E * max|score| < 2^61
  float mx = 0.f;
  for (int i = threadIdx.x; i < E; i += blockDim.x) {
    const int j = i / kk, r = i - j * kk;
    mx = fmaxf(mx, fabsf(key_score(tk[(size_t)j * a.k_max + r])));
  }
  mx = block_max(mx, red);
  int xexp = 0;
  if (mx > 0.f) {
    int e;
    frexpf(mx, &e);                       // mx < 2^e
    const int c = (E > 1) ? 32 - __clz(E - 1) : 0;  // E <= 2^c
    xexp = min(120, max(-120, 61 - e - c));
  }
  for (int f = threadIdx.x; f < F; f += blockDim.x) {
    votes[f] = 0;
    massfx[f] = 0;
  }
  __threadfence();
  __syncthreads();
  for (int i = threadIdx.x; i < E; i += blockDim.x) {
    const int j = i / kk, r = i - j * kk;
    const uint64_t key = tk[(size_t)j * a.k_max + r];
    const int f = frame_of(a, s, key_row(key));
    const long long fx = llrint(ldexp((double)key_score(key), xexp));
    atomicAdd(&votes[f], 1);
    atomicAdd(reinterpret_cast<unsigned long long*>(&massfx[f]), (unsigned long long)fx);
  }
  __threadfence();
  __syncthreads();
  const double inv = ldexp(1.0, -xexp);
  // compact voted frames (frame order) into records: hi = votes:32 | mass_hi:32,
  // lo = mass_lo:32 | ~frame:32, compared descending
  uint64_t* rh = a.rec_hi + (size_t)s * a.f_max;
  uint64_t* rl = a.rec_lo + (size_t)s * a.f_max;
  int n_voted = 0;
  for (int b0 = 0; b0 < F; b0 += blockDim.x) {
    const int f = b0 + threadIdx.x;
    int v = 0;
    int64_t mf = 0;
    if (f < F) {
      v = __hip_atomic_load(&votes[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      mf = __hip_atomic_load(&massfx[f], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a.dbg_vote_hist) {
        a.dbg_vote_hist[(size_t)s * a.hist_stride + f] = v;
        a.dbg_mass_hist[(size_t)s * a.hist_stride + f] = (float)((double)mf * inv);
      }
    }
    const bool p = v >= 1;
    int tot;
    const int pre = block_excl_scan(p ? 1 : 0, scan_sh, tot);
    if (p) {
      const uint64_t mb = (uint64_t)mf ^ 0x8000000000000000ull;
      rh[n_voted + pre] = ((uint64_t)(uint32_t)v << 32) | (mb >> 32);
      rl[n_voted + pre] = (mb << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)f);
    }
    n_voted += tot;
  }
  if (a.dbg_vote_hist) {
    for (int f = F + threadIdx.x; f < a.hist_stride; f += blockDim.x) {
      a.dbg_vote_hist[(size_t)s * a.hist_stride + f] = 0;
      a.dbg_mass_hist[(size_t)s * a.hist_stride + f] = 0.f;
    }
  }
  __threadfence();
  __syncthreads();
  // top `pool` records: rounds of bitonic sorting, the running best kept in front
  const int P = a.pool;
  int kept = 0;
  int next = 0;
  do {
    const int room = kPoolSort - kept;
    const int take = min(room, n_voted - next);
    const int tot = kept + take;
    const int np = pow2_ceil(max(tot, 2));
    for (int i = threadIdx.x; i < take; i += blockDim.x) {
      shi[kept + i] = __hip_atomic_load(&rh[next + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      slo[kept + i] = __hip_atomic_load(&rl[next + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int i = tot + threadIdx.x; i < np; i += blockDim.x) { shi[i] = 0; slo[i] = 0; }
    __syncthreads();
    bitonic_desc_u128(shi, slo, np);
    kept = min(P, tot);
    next += take;
  } while (next < n_voted);
  const int pn = kept;
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    int id = -1, v = 0;
    float m = 0.f;
    if (i < pn) {
      id = (int)(0xFFFFFFFFu - (uint32_t)slo[i]);
      v = (int)(shi[i] >> 32);
      const uint64_t mb = (shi[i] << 32) | (slo[i] >> 32);
      m = (float)((double)(int64_t)(mb ^ 0x8000000000000000ull) * inv);
    }
    a.pool_ids[(size_t)s * P + i] = id;
    a.pool_votes[(size_t)s * P + i] = v;
    a.pool_mass[(size_t)s * P + i] = m;
    if (a.dbg_pool) a.dbg_pool[(size_t)s * P + i] = id;
  }
  if (threadIdx.x == 0) {
    a.pool_n[s] = pn;
    if (a.dbg_pool_n) a.dbg_pool_n[s] = pn;
  }
}

// ---------------------------------------------------------------------------
// k_gram: fp32 Gram matrix of the pool descriptors; 16 x 16 tiles
// ---------------------------------------------------------------------------
struct GramArgs {
  int pool, dim, tiles;
  const float* desc[kMaxStreams];
  const int32_t* pool_ids;
  const int32_t* pool_n;
  float* gram;          // [S][pool][pool]
};

__global__ __launch_bounds__(256) void k_gram(GramArgs a) {
  __shared__ float xi[16][65];
  __shared__ float xj[16][65];
  const int s = blockIdx.x / (a.tiles * a.tiles);
  const int t = blockIdx.x % (a.tiles * a.tiles);
  const int ti = t / a.tiles, tj = t % a.tiles;
  const int pn = a.pool_n[s];
  if (ti * 16 >= pn || tj * 16 >= pn) return;
  const int r = threadIdx.x >> 4, c = threadIdx.x & 15;
  const int32_t* ids = a.pool_ids + (size_t)s * a.pool;
  const float* D = a.desc[s];
  float acc = 0.f;
  for (int e0 = 0; e0 < a.dim; e0 += 64) {
    for (int i = threadIdx.x; i < 16 * 64; i += blockDim.x) {
      const int rr = i >> 6, ee = i & 63;
      const int pi = ti * 16 + rr, pj = tj * 16 + rr;
      const bool ein = e0 + ee < a.dim;
      xi[rr][ee] = (pi < pn && ein) ? D[(size_t)ids[pi] * a.dim + e0 + ee] : 0.f;
      xj[rr][ee] = (pj < pn && ein) ? D[(size_t)ids[pj] * a.dim + e0 + ee] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int e = 0; e < 64; ++e) acc = fmaf(xi[r][e], xj[c][e], acc);
    __syncthreads();
  }
  const int pi = ti * 16 + r, pj = tj * 16 + c;
  if (pi < pn && pj < pn) a.gram[((size_t)s * a.pool + pi) * a.pool + pj] = acc;
}

// ---------------------------------------------------------------------------
// k_maxmin: greedy max-min diversity (one block per stream)
// ---------------------------------------------------------------------------
struct MaxminArgs {
  int pool, n_select;
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

__global__ __launch_bounds__(256) void k_maxmin(MaxminArgs a) {
  __shared__ float mind[kMaxPool];
  __shared__ int taken[kMaxPool];
  __shared__ int sel[kMaxSelect];
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int s = blockIdx.x;
  const int pn = a.pool_n[s];
  const int K = min(a.n_select, pn);
  const float* G = a.gram + (size_t)s * a.pool * a.pool;
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
      mind[u] = fminf(mind[u], 1.0f - G[(size_t)w * a.pool + u]);
      if (u == w) taken[u] = 1;
    }
    if (threadIdx.x == 0) sel[it] = w;
    __syncthreads();
  }
  for (int i = threadIdx.x; i < a.n_select; i += blockDim.x) {
    const size_t o = (size_t)s * a.n_select + i;
    if (i < K) {
      const int p = sel[i];
      a.out_ids[o] = a.pool_ids[(size_t)s * a.pool + p];
      a.out_votes[o] = a.pool_votes[(size_t)s * a.pool + p];
      a.out_mass[o] = a.pool_mass[(size_t)s * a.pool + p];
    } else {
      a.out_ids[o] = -1;
      a.out_votes[o] = 0;
      a.out_mass[o] = 0.f;
    }
  }
  if (threadIdx.x == 0) a.out_n[s] = K;
}

// ---------------------------------------------------------------------------
// Append kernels
// ---------------------------------------------------------------------------
// Descriptor (Eq. memory_key): fp32 mean over the frame's raw last-layer tokens,
// heads flattened head-major, L2-normalised.  Also writes the frame offsets.
template <int D>
__global__ __launch_bounds__(256) void k_desc(AppendArgs a) {
  __shared__ float red[8];
  const int f = blockIdx.x;
  const int T = a.n_tokens, dim = a.Hk * D;
  const int64_t nT = (int64_t)a.n_frames * T;
  const uint16_t* src = a.src[a.L - 1];
  float vals[4];
  float ss = 0.f;
  for (int k = 0; k < 4; ++k) {
    const int e = threadIdx.x + k * 256;
    vals[k] = 0.f;
    if (e < dim) {
      const int g = e / D, ee = e % D;
      const uint16_t* p = src + ((int64_t)g * nT + (int64_t)f * T) * D + ee;
      float acc = 0.f;
      for (int t = 0; t < T; ++t) acc += __uint_as_float((uint32_t)p[(int64_t)t * D] << 16);
      vals[k] = acc / (float)T;
      ss = fmaf(vals[k], vals[k], ss);
    }
  }
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
// mean, then n_iters Lloyd rounds on squared Euclidean distance in fp32.
// One thread per token; centroids in LDS (read as broadcasts).
template <int D>
__global__ __launch_bounds__(256) void k_kmeans(AppendArgs a) {
  constexpr int XS = D / 2 + 1;  // padded row stride in 32-bit words (bank-conflict free)
  __shared__ uint32_t xs[kMaxTokensCompress * XS];
  __shared__ float cen[kMaxCentroids * D];
  __shared__ float mu[D];
  __shared__ float mind[kMaxTokensCompress];
  __shared__ int assign_[kMaxTokensCompress];
  __shared__ int members[kMaxTokensCompress];
  __shared__ int ccount[kMaxCentroids];
  __shared__ int coff[kMaxCentroids];
  __shared__ int chosen[kMaxCentroids];
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int b = blockIdx.x;
  const int g = b % a.Hk, fl = b / a.Hk, l = fl % a.L, f = fl / a.L;
  const int T = a.n_tokens, C = min(a.n_centroids, T);
  const int64_t nT = (int64_t)a.n_frames * T;
  const uint16_t* src = a.src[l] + ((int64_t)g * nT + (int64_t)f * T) * D;
  const int t = threadIdx.x;
  for (int i = t; i < T * (D / 2); i += blockDim.x) {
    const int r = i / (D / 2), w = i % (D / 2);
    xs[r * XS + w] = reinterpret_cast<const uint32_t*>(src + (int64_t)r * D)[w];
  }
  __syncthreads();
  auto xval = [&](int r, int e) -> float {
    const uint32_t w = xs[r * XS + (e >> 1)];
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  };
  // frame mean (token order)
  for (int e = t; e < D; e += blockDim.x) {
    float acc = 0.f;
    for (int r = 0; r < T; ++r) acc += xval(r, e);
    mu[e] = acc / (float)T;
  }
  __syncthreads();
  float dm = -INFINITY;
  if (t < T) {
    float acc = 0.f;
    for (int e = 0; e < D; ++e) { const float d = xval(t, e) - mu[e]; acc = fmaf(d, d, acc); }
    dm = acc;
  }
  int pick = block_argmax(dm, t < T ? t : INT_MAX, shv, shi);
  bool is_taken = (t == pick);
  if (t == 0) chosen[0] = pick;
  float my_min = INFINITY;
  for (int c = 0; c < C; ++c) {
    if (c > 0) {
      pick = block_argmax((t < T && !is_taken) ? my_min : -INFINITY, (t < T && !is_taken) ? t : INT_MAX,
                          shv, shi);
      if (t == pick) is_taken = true;
      if (t == 0) chosen[c] = pick;
    }
    if (t < T) {
      float acc = 0.f;
      for (int e = 0; e < D; ++e) { const float d = xval(t, e) - xval(pick, e); acc = fmaf(d, d, acc); }
      my_min = fminf(my_min, acc);
    }
  }
  __syncthreads();
  for (int i = t; i < C * D; i += blockDim.x) cen[i] = xval(chosen[i / D], i % D);
  __syncthreads();
  for (int it = 0; it < a.n_iters; ++it) {
    // assignment: nearest centre, ties to the lower index
    if (t < T) {
      float acc[kMaxCentroids];
#pragma unroll
      for (int c = 0; c < kMaxCentroids; ++c) acc[c] = 0.f;
      for (int e = 0; e < D; e += 2) {
        const uint32_t w = xs[t * XS + (e >> 1)];
        const float x0 = bf16_lo(w), x1 = bf16_hi(w);
#pragma unroll
        for (int c = 0; c < kMaxCentroids; ++c) {
          if (c < C) {
            const float d0 = x0 - cen[c * D + e], d1 = x1 - cen[c * D + e + 1];
            acc[c] = fmaf(d1, d1, fmaf(d0, d0, acc[c]));
          }
        }
      }
      int bi = 0;
      float bv = acc[0];
#pragma unroll
      for (int c = 1; c < kMaxCentroids; ++c) {
        if (c < C && acc[c] < bv) { bv = acc[c]; bi = c; }
      }
      assign_[t] = bi;
    }
    if (t < kMaxCentroids) ccount[t] = 0;
    __syncthreads();
    // stable counting sort of tokens by centre
    int rank = 0;
    if (t < T) {
      const int me = assign_[t];
      for (int r = 0; r < t; ++r) rank += (assign_[r] == me);
      atomicAdd(&ccount[me], 1);
    }
    __syncthreads();
    if (t == 0) {
      int run = 0;
      for (int c = 0; c < C; ++c) { coff[c] = run; run += ccount[c]; }
    }
    __syncthreads();
    if (t < T) members[coff[assign_[t]] + rank] = t;
    __syncthreads();
    // update: mean of members in token order; empty centres stay
    for (int i = t; i < C * D; i += blockDim.x) {
      const int c = i / D, e = i % D;
      const int n = ccount[c];
      if (n > 0) {
        float acc = 0.f;
        for (int q = 0; q < n; ++q) acc += xval(members[coff[c] + q], e);
        cen[i] = acc / (float)n;
      }
    }
    __syncthreads();
  }
  const int64_t drow0 = ((int64_t)l * a.Hk + g) * a.max_rows + a.row0 + (int64_t)f * C;
  for (int i = t; i < C * D; i += blockDim.x) {
    a.dst.keys[(drow0 + i / D) * D + (i % D)] = bf16_rne(cen[i]);
  }
  for (int c = t; c < C; c += blockDim.x) a.dst.counts[drow0 + c] = a.n_iters > 0 ? ccount[c] : 0;
}

inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

template <int D>
hipError_t append_impl(const AppendArgs& a, bool compress, hipStream_t st) {
  hipLaunchKernelGGL(k_desc<D>, dim3(a.n_frames), dim3(256), 0, st, a);
  if (compress) {
    hipLaunchKernelGGL(k_kmeans<D>, dim3(a.n_frames * a.L * a.Hk), dim3(256), 0, st, a);
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
    a.item_base[s] = items;
    items += p.L * p.ngs * cdiv(a.units[s], a.chunk);
    a.full_base[s] = p.full_base[s];
    a.full_stride[s] = p.st[s].n;
  }
  a.item_base[p.S] = items;
  a.total_items = items;
  a.samp = p.samp; a.samp_stride = p.m_max;
  a.tau = p.tau; a.cnt = p.cnt; a.cand = p.cand; a.cap = p.cap;
  a.flag = p.flag; a.only_list = -1; a.full = p.full; a.row0 = 0;
  return a;
}

template <int D, int KIND>
void launch_score(const ScoreArgs& a, int head_mode, int max_grid, hipStream_t st) {
  if (a.total_items == 0) return;
  const int grid = std::min(a.total_items, max_grid);
  if (head_mode == 0) hipLaunchKernelGGL((k_score<D, KIND>), dim3(grid), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((k_score_hm<D, KIND>), dim3(grid), dim3(256), 0, st, a);
}

template <int D>
hipError_t retrieve_impl(RetrievePlan& p, hipStream_t st) {
  // 1. query prep
  {
    const int pairs = p.S * p.L;
    for (int first = 0; first < pairs; first += 128) {
      PrepArgs a{};
      a.Hq = p.Hq; a.Hk = p.Hk; a.G = p.G; a.L = p.L; a.head_mode = p.head_mode; a.first = first;
      const int cnt = std::min(128, pairs - first);
      for (int i = 0; i < cnt; ++i) {
        const int pr = first + i;
        a.q[i] = p.st[pr / p.L].q[pr % p.L];
      }
      for (int s = 0; s < p.S; ++s) { a.nq[s] = p.st[s].nq; a.qscale[s] = p.st[s].qscale; }
      a.qB = reinterpret_cast<u32x4*>(p.qB);
      hipLaunchKernelGGL(k_prep<D>, dim3(cnt * p.Hk), dim3(64), 0, st, a);
    }
  }
  ListArgs la{};
  la.NL = p.NL; la.S = p.S; la.cap = p.cap; la.k_max = p.k_max; la.top_k = p.top_k;
  for (int s = 0; s < p.S; ++s) {
    la.m[s] = p.st[s].m; la.r[s] = p.st[s].r; la.kk[s] = p.st[s].kk; la.n[s] = p.st[s].n;
    la.full_base[s] = p.full_base[s];
  }
  la.samp = p.samp; la.samp_stride = p.m_max; la.tau = p.tau; la.cnt = p.cnt; la.flag = p.flag;
  la.cand = p.cand; la.topk = p.topk; la.full = p.full;
  la.dbg_pos = p.dbg_topk_pos; la.dbg_score = p.dbg_topk_score; la.dbg_stats = p.dbg_list_stats;
  const int lists = p.S * p.NL;
  // 2. sample scores, 3. thresholds
  launch_score<D, K_SAMPLE>(make_score_args(p, K_SAMPLE), p.head_mode, 4096, st);
  hipLaunchKernelGGL(k_thresh, dim3(lists), dim3(256), 0, st, la);
  // 4. streaming pass over every key row
  if (p.ev_start) (void)hipEventRecord(p.ev_start, st);
  launch_score<D, K_STREAM>(make_score_args(p, K_STREAM), p.head_mode, 2048, st);
  if (p.ev_stop) (void)hipEventRecord(p.ev_stop, st);
  // 5. exact top-k from candidates; 6. exact fallback for flagged lists
  hipLaunchKernelGGL(k_select, dim3(lists), dim3(256), 0, st, la);
  launch_score<D, K_FULL>(make_score_args(p, K_FULL), p.head_mode, 1024, st);
  hipLaunchKernelGGL(k_fb_select, dim3(lists), dim3(256), 0, st, la);
  // 7. votes, mass and pool
  VoteArgs va{};
  va.NL = p.NL; va.k_max = p.k_max; va.pool = p.pool; va.f_max = p.f_max;
  va.hist_stride = p.dbg_hist_stride;
  for (int s = 0; s < p.S; ++s) {
    va.kk[s] = p.st[s].kk; va.f[s] = p.st[s].f; va.rpf[s] = p.st[s].rpf;
    va.frame_off[s] = p.st[s].frame_off;
  }
  va.topk = p.topk; va.votes_g = p.votes; va.massfx_g = p.massfx;
  va.rec_hi = p.rec_hi; va.rec_lo = p.rec_lo;
  va.pool_ids = p.pool_ids; va.pool_votes = p.pool_votes; va.pool_mass = p.pool_mass;
  va.pool_n = p.pool_n;
  va.dbg_vote_hist = p.dbg_vote_hist; va.dbg_mass_hist = p.dbg_mass_hist;
  va.dbg_pool = p.dbg_pool; va.dbg_pool_n = p.dbg_pool_n;
  hipLaunchKernelGGL(k_votes_pool, dim3(p.S), dim3(1024), 0, st, va);
  // 8. Gram matrix, 9. max-min
  GramArgs ga{};
  ga.pool = p.pool; ga.dim = p.Hk * D; ga.tiles = cdiv(p.pool, 16);
  for (int s = 0; s < p.S; ++s) ga.desc[s] = p.st[s].desc;
  ga.pool_ids = p.pool_ids; ga.pool_n = p.pool_n; ga.gram = p.gram;
  hipLaunchKernelGGL(k_gram, dim3(p.S * ga.tiles * ga.tiles), dim3(256), 0, st, ga);
  MaxminArgs ma{};
  ma.pool = p.pool; ma.n_select = p.n_select;
  ma.pool_ids = p.pool_ids; ma.pool_votes = p.pool_votes; ma.pool_mass = p.pool_mass;
  ma.pool_n = p.pool_n; ma.gram = p.gram;
  ma.out_ids = p.out_ids; ma.out_votes = p.out_votes; ma.out_mass = p.out_mass; ma.out_n = p.out_n;
  hipLaunchKernelGGL(k_maxmin, dim3(p.S), dim3(256), 0, st, ma);
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
  hipLaunchKernelGGL(k_prep<D>, dim3(p.L * p.Hk), dim3(64), 0, st, pa);
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
  a.flag = nullptr;
  a.only_list = p.head_mode == 0 ? layer * p.Hq + q_head : layer;
  a.full = out; a.full_base[0] = -(int64_t)a.only_list * n_rows; a.full_stride[0] = (int32_t)n_rows;
  a.row0 = row0;
  if (n_rows > 0) launch_score<D, K_FULL>(a, p.head_mode, 2048, st);
  return hipGetLastError();
}

}  // namespace

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
  p.flag = static_cast<int32_t*>(take(lists * 4));
  p.samp = static_cast<float*>(take(lists * (size_t)p.m_max * 4));
  p.cand = static_cast<uint64_t*>(take(lists * (size_t)p.cap * 8));
  p.topk = static_cast<uint64_t*>(take(lists * (size_t)std::max(p.k_max, 1) * 8));
  p.full = static_cast<float*>(take((size_t)p.full_total * 4));
  p.votes = static_cast<int32_t*>(take((size_t)p.S * p.f_max * 4));
  p.massfx = static_cast<int64_t*>(take((size_t)p.S * p.f_max * 8));
  p.rec_hi = static_cast<uint64_t*>(take((size_t)p.S * p.f_max * 8));
  p.rec_lo = static_cast<uint64_t*>(take((size_t)p.S * p.f_max * 8));
  p.pool_ids = static_cast<int32_t*>(take((size_t)p.S * p.pool * 4));
  p.pool_votes = static_cast<int32_t*>(take((size_t)p.S * p.pool * 4));
  p.pool_mass = static_cast<float*>(take((size_t)p.S * p.pool * 4));
  p.pool_n = static_cast<int32_t*>(take((size_t)p.S * 4));
  p.gram = static_cast<float*>(take((size_t)p.S * p.pool * p.pool * 4));
  return (off + 255) & ~(size_t)255;
}

hipError_t launch_append(const AppendArgs& a, bool compress, hipStream_t st) {
  return a.D == 128 ? append_impl<128>(a, compress, st) : append_impl<64>(a, compress, st);
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
