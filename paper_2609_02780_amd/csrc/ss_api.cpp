// C ABI of the shallow-index evidence retrieval library: argument validation,
// per-index host bookkeeping and the retrieval planner.  Every check runs before
// any HIP call, so invalid calls leave the index and the device untouched.
#include "../../include/shallowstream.h"
#include "ss_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

struct ss_index {
  ss_index_desc desc;
  void* arena;
  size_t arena_bytes;
  ss::IndexDev dev;
  int64_t n_frames;          // frames appended so far: ids 0 .. n_frames - 1
  int64_t frame_base = 0;    // frames below it were dropped from the arena (ss_index_compact);
                             // per-frame arena entries are indexed by id - frame_base
  int64_t n_rows;            // rows the arena holds per (layer, KV head)
  std::vector<int64_t> off;  // arena row offsets of frames frame_base .. n_frames
  int64_t first_detail = 0;  // frames before it were folded into long-term clusters
  int32_t rpf;               // common rows per frame, 0 if mixed, -1 before the first append
};

namespace {

// The last failure's text: a fixed buffer, so recording an error never allocates.
thread_local char g_err[512] = "";
thread_local hipEvent_t g_ev_start = nullptr;
thread_local hipEvent_t g_ev_stop = nullptr;

ss_status fail(ss_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

// Runs the body of an entry point; no C++ exception crosses the C ABI (host
// allocations can throw std::bad_alloc).
template <class F>
ss_status guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(SS_ERR_INTERNAL, "out of host memory");
  } catch (...) {
    return fail(SS_ERR_INTERNAL, "unexpected C++ exception");
  }
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct Layout {
  size_t keys, counts, desc, pooled, off, stats, total;
};

// Check an index shape; fills `why` on failure.
ss_status check_desc(const ss_index_desc* d) {
  if (!d) return fail(SS_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->n_layers < 1 || d->n_layers > ss::kMaxLayers)
    return fail(SS_ERR_UNSUPPORTED, "n_layers %d outside 1..%d", d->n_layers, ss::kMaxLayers);
  if (d->n_q_heads < 1 || d->n_kv_heads < 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "head counts must be >= 1");
  if (d->n_q_heads % d->n_kv_heads != 0)
    return fail(SS_ERR_INVALID_ARGUMENT, "n_q_heads %d is not a multiple of n_kv_heads %d",
                d->n_q_heads, d->n_kv_heads);
  if (d->n_q_heads / d->n_kv_heads > ss::kMaxGroup)
    return fail(SS_ERR_UNSUPPORTED, "query heads per KV head %d > %d",
                d->n_q_heads / d->n_kv_heads, ss::kMaxGroup);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SS_ERR_UNSUPPORTED, "head_dim %d is not 64 or 128", d->head_dim);
  if ((int64_t)d->n_kv_heads * d->head_dim > 1024)
    return fail(SS_ERR_UNSUPPORTED, "n_kv_heads * head_dim %lld > 1024",
                (long long)d->n_kv_heads * d->head_dim);
  if (d->max_frames < 1 || d->max_frames > (int64_t)1 << 30)
    return fail(SS_ERR_INVALID_ARGUMENT, "max_frames %lld outside 1..2^30", (long long)d->max_frames);
  if (d->max_rows < 1 || d->max_rows > (int64_t)0x7FFFFFFF - 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "max_rows %lld outside 1..2^31-2", (long long)d->max_rows);
  // one (layer, KV head) segment is read through a 32-bit buffer range
  if (d->max_rows * d->head_dim * 2 > ((int64_t)1 << 31) - 1)
    return fail(SS_ERR_UNSUPPORTED, "max_rows * head_dim * 2 = %lld bytes per (layer, KV head) >= 2^31",
                (long long)(d->max_rows * d->head_dim * 2));
  if (d->n_recent < 0) return fail(SS_ERR_INVALID_ARGUMENT, "n_recent must be >= 0");
  if ((int64_t)d->n_layers * d->n_q_heads > ss::kMaxListsPerStream)
    return fail(SS_ERR_UNSUPPORTED, "n_layers * n_q_heads %lld > %d",
                (long long)d->n_layers * d->n_q_heads, ss::kMaxListsPerStream);
  return SS_OK;
}

Layout layout(const ss_index_desc& d) {
  Layout L{};
  const size_t lg = (size_t)d.n_layers * d.n_kv_heads;
  size_t off = 0;
  L.keys = off;
  off = align256(off + lg * (size_t)d.max_rows * d.head_dim * 2);
  L.counts = off;
  off = align256(off + lg * (size_t)d.max_rows * 4);
  L.desc = off;
  off = align256(off + (size_t)d.max_frames * d.n_kv_heads * d.head_dim * 4);
  L.pooled = off;
  off = align256(off + (size_t)d.max_frames * lg * d.head_dim * 4);
  L.off = off;
  off = align256(off + ((size_t)d.max_frames + 1) * 4);
  L.stats = off;
  off = align256(off + 16);
  L.total = off;
  return L;
}

bool same_shape(const ss_index_desc& a, const ss_index_desc& b) {
  return a.n_layers == b.n_layers && a.n_q_heads == b.n_q_heads && a.n_kv_heads == b.n_kv_heads &&
         a.head_dim == b.head_dim;
}

// Candidate frames [f_lo, f_hi) and rows [r_lo, r_hi) of an index: Eq.
// context_partition excludes the newest n_recent frames, and with long-history
// compression the frames already folded into clusters are not token candidates
// (the detailed history S_T of Eq. optional_context_compression).
struct Window {
  int64_t f_lo, f_hi, r_lo, r_hi;
};
// Arena row where frame f's rows start (frame_base <= f <= n_frames).
inline int64_t row_of(const ss_index* x, int64_t f) { return x->off[(size_t)(f - x->frame_base)]; }

Window candidates(const ss_index* x) {
  Window w;
  // frames leave the arena only after they left the detailed window, which
  // never reaches into the recent window: frame_base <= f_lo <= f_hi
  w.f_hi = std::max(x->frame_base, x->n_frames - x->desc.n_recent);
  w.f_lo = std::min(x->first_detail, w.f_hi);
  w.r_lo = row_of(x, w.f_lo);
  w.r_hi = row_of(x, w.f_hi);
  return w;
}

constexpr int kSampleRank = 32;      // rank r of the sample cut-off
constexpr int kFullScanRows = 4096;  // at or below this many rows the sample is the whole list
static_assert(kFullScanRows <= 16384, "a full-scan sample must fit the register select");
constexpr int kChunkRows = 4096;
constexpr int kSampleChunk = 128;

// Expected candidates per list: 6k (at least 1024), raised for very long lists
// so the sample stays within the register select (kSampleMax rows).  The count
// behaves like E Gamma(r) / r; it falls below k with probability
// P(Poisson(r k / E) >= r) and exceeds the capacity 3E with probability
// P(Poisson(3 r) <= r - 1); either case takes the exact fallback.  A smaller E
// keeps fewer tiles on the candidate path of the streaming pass and fewer
// candidates for the selection; a larger E allows a smaller r, hence a smaller
// sample (m = r n / E).  E = 6k gives r = 14, where the capacity tail binds
// (m = 3,216 of 705,600 rows per list group on the 1-hour index); against 4k
// (r = 21) it took 2 to 7 us off a call on the 1-hour, paper-settings, 10-minute
// and 16-stream workloads, and 8k was slower on all four.
constexpr int64_t kSampleMax = 16384;
int64_t expected_candidates(int64_t n, int64_t kk) {
  const int64_t r = std::min<int64_t>(kk, kSampleRank);
  return std::max<int64_t>({6 * kk, 1024, (n * r + kSampleMax - 1) / kSampleMax});
}

// P(X >= r) for X ~ Poisson(lam): the terms from r upward, in log space.
double poisson_tail(double lam, int r) {
  if (lam <= 0.0) return r <= 0 ? 1.0 : 0.0;
  double term = std::exp(-lam + r * std::log(lam) - std::lgamma(r + 1.0)), sum = 0.0;
  for (int i = r; i < r + 2000 && term > 1e-300; ++i) {
    sum += term;
    term *= lam / (i + 1);
  }
  return sum;
}

// P(X <= r) for X ~ Poisson(lam).
double poisson_cdf(double lam, int r) {
  if (r < 0) return 0.0;
  double term = std::exp(-lam), sum = 0.0;
  for (int i = 0; i <= r; ++i) {
    sum += term;
    term *= lam / (i + 1);
  }
  return std::min(sum, 1.0);
}

// The smallest sample rank r <= min(k, 32) whose chances of too few candidates,
// P(Poisson(r k / E) >= r), and of more than the capacity (at least 3E),
// P(Poisson(3 r) <= r - 1), are both at most kFallbackOdds per list.
constexpr double kFallbackOdds = 2e-7;
int64_t sample_rank(int64_t kk, int64_t E) {
  const int64_t rmax = std::min<int64_t>(kk, kSampleRank);
  for (int64_t r = 1; r < rmax; ++r)
    if (poisson_tail((double)r * (double)kk / (double)E, (int)r) <= kFallbackOdds &&
        poisson_cdf(3.0 * (double)r, (int)r - 1) <= kFallbackOdds)
      return r;
  return rmax;
}

struct StreamSizes {
  int n, f, m, r, kk;
};

// Sample plan of one list.  With m sampled rows spread evenly over n rows and the
// cut-off at the r-th largest sample score, about r n / m rows score at or above
// it (the expected candidate count E).  r from sample_rank (14 when E = 6k);
// m = n gives an exact cut (r = k) for small lists.
StreamSizes plan_stream(int64_t n, int64_t f, int top_k) {
  StreamSizes z{};
  z.n = (int)n;
  z.f = (int)f;
  z.kk = (int)std::min<int64_t>(top_k, n);
  if (n == 0) return z;
  const int64_t E = expected_candidates(n, z.kk);
  int64_t r = sample_rank(z.kk, E);
  int64_t m = std::max<int64_t>(r, (n * r + E - 1) / E);
  if (n <= kFullScanRows || (2 * m >= n && n <= kSampleMax)) {
    m = n;
    r = z.kk;
  }
  z.m = (int)m;
  z.r = (int)r;
  return z;
}

int64_t candidate_cap(int top_k, int64_t n_max) {
  const int64_t kk = std::min<int64_t>(top_k, std::max<int64_t>(n_max, 1));
  return std::max<int64_t>(3 * expected_candidates(n_max, kk), 4096);
}

ss_status check_params(const ss_retrieve_params* p, int Hk, int D) {
  if (!p) return fail(SS_ERR_INVALID_ARGUMENT, "params is NULL");
  if (p->top_k < 1 || p->top_k > ss::kMaxTopK)
    return fail(SS_ERR_UNSUPPORTED, "top_k %d outside 1..%d", p->top_k, ss::kMaxTopK);
  if (p->n_select < 1 || p->n_select > ss::kMaxSelect)
    return fail(SS_ERR_UNSUPPORTED, "n_select %d outside 1..%d", p->n_select, ss::kMaxSelect);
  if (p->pool_mult < 1) return fail(SS_ERR_INVALID_ARGUMENT, "pool_mult must be >= 1");
  if ((int64_t)p->pool_mult * p->n_select > ss::kMaxPool)
    return fail(SS_ERR_UNSUPPORTED, "pool_mult * n_select %lld > %d",
                (long long)p->pool_mult * p->n_select, ss::kMaxPool);
  if (p->head_mode != 0 && p->head_mode != 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "head_mode must be 0 or 1");
  if (p->head_mode == 1 && Hk > 8)
    return fail(SS_ERR_UNSUPPORTED, "head_mode 1 supports at most 8 KV heads");
  if (p->score_mode != 0 && p->score_mode != 1)
    return fail(SS_ERR_INVALID_ARGUMENT, "score_mode must be 0 or 1");
  if (p->head_mode == 1 && p->score_mode == 1 &&
      ((int64_t)Hk * D > 512 || (Hk != 1 && Hk != 2 && Hk != 4 && Hk != 8)))
    return fail(SS_ERR_UNSUPPORTED,
                "head_mode 1 with attention probabilities needs n_kv_heads in {1, 2, 4, 8} and "
                "n_kv_heads * head_dim <= 512");
  return SS_OK;
}

// Builds the plan of streams [s0, s0 + S) of a validated batch (`queries` may be
// NULL when only the workspace size is wanted).
void build_plan(ss::RetrievePlan& p, ss_index* const* idx, int s0, int S, const void* const* queries,
                const int32_t* n_q, const ss_retrieve_params* prm) {
  std::memset(&p, 0, sizeof p);
  const ss_index_desc& d = idx[0]->desc;
  p.S = S;
  p.L = d.n_layers;
  p.Hq = d.n_q_heads;
  p.Hk = d.n_kv_heads;
  p.G = p.Hq / p.Hk;
  p.D = d.head_dim;
  p.head_mode = prm->head_mode;
  p.score_mode = prm->score_mode;
  p.hm_prob = prm->head_mode == 1 && prm->score_mode == 1;
  p.NL = prm->head_mode == 0 ? p.L * p.Hq : p.L;
  p.NLs = p.hm_prob ? p.L * p.Hq : p.NL;
  p.ncol = prm->head_mode == 0 ? p.G : 1;
  p.ngs = prm->head_mode == 0 ? p.Hk : 1;
  p.top_k = prm->top_k;
  p.n_select = prm->n_select;
  p.pool_mult = prm->pool_mult;
  p.pool = prm->pool_mult * prm->n_select;
  p.chunk_rows = kChunkRows;
  p.samp_chunk = kSampleChunk;
  int64_t n_max = 0;
  int hist = 1;
  for (int i = 0; i < S; ++i) {
    const ss_index* x = idx[s0 + i];
    const Window w = candidates(x);
    const int64_t rows = w.r_hi - w.r_lo, frames = w.f_hi - w.f_lo;
    const StreamSizes z = plan_stream(rows, frames, prm->top_k);
    ss::StreamPlan& sp = p.st[i];
    sp.keys = x->dev.keys + w.r_lo * d.head_dim;          // each (layer, KV head) run from r_lo
    sp.frame_off = x->dev.frame_off + (w.f_lo - x->frame_base);
    sp.desc = x->dev.desc + (w.f_lo - x->frame_base) * (int64_t)d.n_kv_heads * d.head_dim;
    sp.frame0 = w.f_lo;
    sp.hist0 = w.f_lo - x->frame_base;
    sp.row0 = w.r_lo;
    sp.kmax = x->dev.stats;
    sp.row_stride = (int32_t)x->desc.max_rows;
    sp.n = z.n;
    sp.f = z.f;
    sp.m = z.m;
    sp.r = z.r;
    sp.kk = z.kk;
    sp.nq = n_q[s0 + i];
    sp.rpf = x->rpf > 0 ? x->rpf : 0;
    double sc = 1.0 / ((double)sp.nq * std::sqrt((double)p.D));
    if (prm->head_mode == 1 && !p.hm_prob) sc /= (double)p.Hq;   // the logit mean folds 1/H_q into the query
    sp.qscale = (float)sc;
    for (int l = 0; l < p.L; ++l)
      sp.q[l] = queries ? static_cast<const uint16_t*>(queries[(size_t)(s0 + i) * p.L + l]) : nullptr;
    n_max = std::max<int64_t>(n_max, rows);
    p.k_max = std::max(p.k_max, z.kk);
    p.m_max = std::max(p.m_max, z.m);
    p.f_max = std::max(p.f_max, z.f);
    hist = (int)std::max<int64_t>(hist, x->desc.max_frames);
  }
  p.f_max = std::max(p.f_max, 1);
  p.m_max = std::max(p.m_max, 1);
  p.cap = (int)candidate_cap(prm->top_k, n_max);
  p.dbg_hist_stride = hist;
}

ss_status check_batch(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                      const ss_retrieve_params* prm) {
  if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
  if (n_streams < 1) return fail(SS_ERR_INVALID_ARGUMENT, "n_streams must be >= 1");
  if (!n_q) return fail(SS_ERR_INVALID_ARGUMENT, "n_q is NULL");
  for (int s = 0; s < n_streams; ++s) {
    if (!idx[s]) return fail(SS_ERR_INVALID_ARGUMENT, "idx[%d] is NULL", s);
    if (!same_shape(idx[s]->desc, idx[0]->desc))
      return fail(SS_ERR_INVALID_ARGUMENT, "idx[%d] shape differs from idx[0]", s);
    if (n_q[s] < 1 || n_q[s] > 4096)
      return fail(SS_ERR_INVALID_ARGUMENT, "n_q[%d] = %d outside 1..4096", s, n_q[s]);
  }
  return check_params(prm, idx[0]->desc.n_kv_heads, idx[0]->desc.head_dim);
}

size_t group_ws(ss_index* const* idx, int s0, int S, const int32_t* n_q,
                const ss_retrieve_params* prm) {
  ss::RetrievePlan p;
  build_plan(p, idx, s0, S, nullptr, n_q, prm);
  return ss::carve_workspace(p, nullptr);
}

size_t batch_ws(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                const ss_retrieve_params* prm) {
  size_t need = 0;
  for (int s0 = 0; s0 < n_streams; s0 += ss::kMaxStreams) {
    const int S = std::min(ss::kMaxStreams, n_streams - s0);
    need = std::max(need, group_ws(idx, s0, S, n_q, prm));
  }
  return need;
}

ss_status retrieve_common(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                          const int32_t* n_q, const ss_retrieve_params* prm, void* ws,
                          size_t ws_bytes, void* stream, int64_t* frame_ids, int32_t* votes,
                          float* mass, int32_t* n_out, const ss_debug_out* dbg) {
  ss_status st = check_batch(idx, n_streams, n_q, prm);
  if (st) return st;
  if (!queries) return fail(SS_ERR_INVALID_ARGUMENT, "queries is NULL");
  const int L = idx[0]->desc.n_layers;
  for (int i = 0; i < n_streams * L; ++i) {
    if (!queries[i]) return fail(SS_ERR_INVALID_ARGUMENT, "queries[%d] is NULL", i);
    if (!aligned(queries[i], 16)) return fail(SS_ERR_INVALID_ARGUMENT, "queries[%d] not 16-byte aligned", i);
  }
  if (!frame_ids || !votes || !mass || !n_out)
    return fail(SS_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
  if (!ws || !aligned(ws, 256)) return fail(SS_ERR_WORKSPACE, "workspace NULL or not 256-byte aligned");
  const size_t need = batch_ws(idx, n_streams, n_q, prm);
  if (ws_bytes < need)
    return fail(SS_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", ws_bytes, need);
  if (dbg && dbg->topk_score == nullptr && dbg->topk_pos != nullptr)
    return fail(SS_ERR_INVALID_ARGUMENT, "debug topk_pos needs topk_score");
  if (dbg && (dbg->vote_hist == nullptr) != (dbg->mass_hist == nullptr))
    return fail(SS_ERR_INVALID_ARGUMENT, "debug vote_hist and mass_hist go together");
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  for (int s0 = 0; s0 < n_streams; s0 += ss::kMaxStreams) {
    const int S = std::min(ss::kMaxStreams, n_streams - s0);
    ss::RetrievePlan p;
    build_plan(p, idx, s0, S, queries, n_q, prm);
    ss::carve_workspace(p, ws);
    p.out_ids = frame_ids + (size_t)s0 * prm->n_select;
    p.out_votes = votes + (size_t)s0 * prm->n_select;
    p.out_mass = mass + (size_t)s0 * prm->n_select;
    p.out_n = n_out + s0;
    p.out_stride = prm->n_select;
    if (dbg) {
      const size_t NLt = (size_t)p.NL * prm->top_k;
      int hist = 1;
      for (int s = 0; s < n_streams; ++s) hist = (int)std::max<int64_t>(hist, idx[s]->desc.max_frames);
      p.dbg_hist_stride = hist;
      p.dbg_topk_pos = dbg->topk_pos ? dbg->topk_pos + (size_t)s0 * NLt : nullptr;
      p.dbg_topk_score = dbg->topk_score ? dbg->topk_score + (size_t)s0 * NLt : nullptr;
      p.dbg_vote_hist = dbg->vote_hist ? dbg->vote_hist + (size_t)s0 * hist : nullptr;
      p.dbg_mass_hist = dbg->mass_hist ? dbg->mass_hist + (size_t)s0 * hist : nullptr;
      p.dbg_pool = dbg->pool ? dbg->pool + (size_t)s0 * p.pool : nullptr;
      p.dbg_pool_n = dbg->pool_n ? dbg->pool_n + s0 : nullptr;
      p.dbg_list_stats = dbg->list_stats ? dbg->list_stats + (size_t)s0 * p.NL * 2 : nullptr;
    }
    p.ev_start = g_ev_start;
    p.ev_stop = g_ev_stop;
    const hipError_t e = ss::launch_retrieve(p, hs);
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "retrieve launch failed: %s", hipGetErrorString(e));
  }
  return SS_OK;
}

// Plan of one group of streams [s0, s0 + S) of a pooled-ranking batch.
void build_pooled(ss::PooledPlan& p, ss_index* const* idx, int s0, int S, const void* const* queries,
                  const int32_t* n_q, int n_select) {
  std::memset(&p, 0, sizeof p);
  const ss_index_desc& d = idx[0]->desc;
  p.S = S; p.L = d.n_layers; p.Hq = d.n_q_heads; p.Hk = d.n_kv_heads; p.G = p.Hq / p.Hk;
  p.D = d.head_dim; p.n_select = n_select;
  for (int i = 0; i < S; ++i) {
    const ss_index* x = idx[s0 + i];
    const Window w = candidates(x);
    const int64_t frames = w.f_hi - w.f_lo;
    p.F[i] = frames;
    p.frame0[i] = w.f_lo;
    p.f_max = std::max<int64_t>(p.f_max, frames);
    p.pooled[i] = x->dev.pooled + (w.f_lo - x->frame_base) * (int64_t)p.L * p.Hk * p.D;
    p.nq[i] = n_q[s0 + i];
    for (int l = 0; l < p.L; ++l)
      p.q[i * p.L + l] = queries ? static_cast<const uint16_t*>(queries[(size_t)(s0 + i) * p.L + l]) : nullptr;
  }
}

size_t pooled_ws(ss_index* const* idx, int32_t n_streams, const int32_t* n_q, int n_select) {
  size_t need = 0;
  for (int s0 = 0; s0 < n_streams; s0 += ss::kMaxStreams) {
    ss::PooledPlan p;
    build_pooled(p, idx, s0, std::min(ss::kMaxStreams, n_streams - s0), nullptr, n_q, n_select);
    need = std::max(need, ss::pooled_workspace(p, nullptr));
  }
  return need;
}

ss_status check_pooled(ss_index* const* idx, int32_t n_streams, const int32_t* n_q, int32_t n_select) {
  if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
  if (n_streams < 1) return fail(SS_ERR_INVALID_ARGUMENT, "n_streams must be >= 1");
  if (!n_q) return fail(SS_ERR_INVALID_ARGUMENT, "n_q is NULL");
  for (int s = 0; s < n_streams; ++s) {
    if (!idx[s]) return fail(SS_ERR_INVALID_ARGUMENT, "idx[%d] is NULL", s);
    if (!same_shape(idx[s]->desc, idx[0]->desc))
      return fail(SS_ERR_INVALID_ARGUMENT, "idx[%d] shape differs from idx[0]", s);
    if (n_q[s] < 1 || n_q[s] > 4096)
      return fail(SS_ERR_INVALID_ARGUMENT, "n_q[%d] = %d outside 1..4096", s, n_q[s]);
  }
  if (n_select < 1 || n_select > ss::kMaxSelect)
    return fail(SS_ERR_UNSUPPORTED, "n_select %d outside 1..%d", n_select, ss::kMaxSelect);
  return SS_OK;
}

struct ClusterLayout {
  size_t state, centroids, sizes, span, reps, total;
};

bool cluster_desc_ok(const ss_cluster_desc* d) {
  return d && d->n_layers >= 1 && d->n_layers <= ss::kMaxLayers && d->n_kv_heads >= 1 &&
         (d->head_dim == 64 || d->head_dim == 128) && (int64_t)d->n_kv_heads * d->head_dim <= 1024 &&
         d->rows_per_unit >= 1 && d->rows_per_unit <= 65536 && d->max_clusters >= 1 &&
         d->max_clusters <= ((int64_t)1 << 30) && std::isfinite(d->tau);
}

ClusterLayout cluster_layout(const ss_cluster_desc& d) {
  ClusterLayout L{};
  const size_t dim = (size_t)d.n_kv_heads * d.head_dim, M = (size_t)d.max_clusters;
  size_t off = 0;
  L.state = off;
  off = align256(off + 16);
  L.centroids = off;
  off = align256(off + M * dim * 4);
  L.sizes = off;
  off = align256(off + M * 4);
  L.span = off;
  off = align256(off + M * 16);
  L.reps = off;
  off = align256(off + M * d.n_layers * dim * d.rows_per_unit * 4);
  L.total = off;
  return L;
}

// Candidate items of one stream's evidence, or -1 for invalid parameters.
int64_t evidence_units_max(const ss_evidence_params* p, int32_t n_select, int32_t k_clusters) {
  if (!p || p->n_recent < 0 || p->n_before < 0 || p->n_after < 0) return -1;
  if (p->retrieved != 0 && p->retrieved != 1) return -1;
  if (k_clusters < 0 || k_clusters > ss::kMaxSelect) return -1;
  int64_t n = p->n_recent;
  if (p->retrieved) {
    if (n_select < 1 || n_select > ss::kMaxSelect) return -1;
    n += (int64_t)n_select * (1 + (int64_t)p->n_before + p->n_after) + k_clusters;
  }
  return n;
}

}  // namespace

struct ss_clusters {
  ss_cluster_desc desc;
  ss::ClusterDev dev;
};

extern "C" {

size_t ss_clusters_required_bytes(const ss_cluster_desc* desc) {
  return cluster_desc_ok(desc) ? cluster_layout(*desc).total : 0;
}

ss_status ss_clusters_create(const ss_cluster_desc* desc, void* dev_arena, size_t arena_bytes, void* stream,
                             ss_clusters** out) {
  return guarded([&]() -> ss_status {
    if (!out) return fail(SS_ERR_INVALID_ARGUMENT, "out is NULL");
    if (!cluster_desc_ok(desc)) return fail(SS_ERR_INVALID_ARGUMENT, "invalid cluster description");
    if (!dev_arena || !aligned(dev_arena, 256)) return fail(SS_ERR_INVALID_ARGUMENT, "arena NULL or not 256-byte aligned");
    const ClusterLayout L = cluster_layout(*desc);
    if (arena_bytes < L.total) return fail(SS_ERR_CAPACITY, "arena %zu bytes, %zu needed", arena_bytes, L.total);
    ss_clusters* c = new (std::nothrow) ss_clusters;
    if (!c) return fail(SS_ERR_INTERNAL, "out of host memory");
    c->desc = *desc;
    char* b = static_cast<char*>(dev_arena);
    c->dev.state = reinterpret_cast<int32_t*>(b + L.state);
    c->dev.centroids = reinterpret_cast<float*>(b + L.centroids);
    c->dev.sizes = reinterpret_cast<int32_t*>(b + L.sizes);
    c->dev.span = reinterpret_cast<int64_t*>(b + L.span);
    c->dev.reps = reinterpret_cast<float*>(b + L.reps);
    const hipError_t e = ss::launch_zero32(c->dev.state, 4, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
      delete c;
      return fail(SS_ERR_DEVICE, "cluster state reset: %s", hipGetErrorString(e));
    }
    *out = c;
    return SS_OK;
  });
}

ss_status ss_clusters_destroy(ss_clusters* cl) {
  return guarded([&]() -> ss_status {
    delete cl;
    return SS_OK;
  });
}

size_t ss_clusters_absorb_workspace_bytes(int64_t n_frames) {
  return n_frames < 0 ? 0 : std::max<size_t>(256, ((size_t)n_frames * 8 + 255) & ~(size_t)255);
}

ss_status ss_clusters_absorb(ss_clusters* cl, ss_index* idx, int64_t frame_hi, void* ws, size_t ws_bytes,
                             void* stream) {
  return guarded([&]() -> ss_status {
    if (!cl || !idx) return fail(SS_ERR_INVALID_ARGUMENT, "cluster set or index is NULL");
    const ss_cluster_desc& c = cl->desc;
    const ss_index_desc& d = idx->desc;
    if (c.n_layers != d.n_layers || c.n_kv_heads != d.n_kv_heads || c.head_dim != d.head_dim)
      return fail(SS_ERR_INVALID_ARGUMENT, "cluster set and index shapes differ");
    const int64_t f_lo = idx->first_detail;
    const int64_t f_end = std::max<int64_t>(0, idx->n_frames - d.n_recent);
    if (frame_hi < f_lo || frame_hi > f_end)
      return fail(SS_ERR_INVALID_ARGUMENT, "frame_hi %lld outside %lld..%lld (frames leave in order, never from the recent window)",
                  (long long)frame_hi, (long long)f_lo, (long long)f_end);
    for (int64_t f = f_lo; f < frame_hi; ++f)
      if (row_of(idx, f + 1) - row_of(idx, f) != c.rows_per_unit)
        return fail(SS_ERR_INVALID_ARGUMENT, "frame %lld stores %lld rows, the cluster set takes %d", (long long)f,
                    (long long)(row_of(idx, f + 1) - row_of(idx, f)), c.rows_per_unit);
    const int64_t n = frame_hi - f_lo;
    if (n > 0x7FFFFFFF) return fail(SS_ERR_UNSUPPORTED, "too many frames in one call");
    if (n > 0 && (!ws || !aligned(ws, 256) || ws_bytes < ss_clusters_absorb_workspace_bytes(n)))
      return fail(SS_ERR_WORKSPACE, "absorb workspace NULL, misaligned or below %zu bytes",
                  ss_clusters_absorb_workspace_bytes(n));
    ss::AbsorbArgs a{};
    a.L = c.n_layers; a.Hk = c.n_kv_heads; a.D = c.head_dim; a.R = c.rows_per_unit;
    a.max_clusters = c.max_clusters; a.max_rows = d.max_rows; a.tau = c.tau;
    a.f_lo = f_lo; a.n_units = (int)n; a.row_lo = row_of(idx, f_lo);
    a.desc = idx->dev.desc + (f_lo - idx->frame_base) * (int64_t)d.n_kv_heads * d.head_dim;
    a.keys = idx->dev.keys;
    a.assign = static_cast<int32_t*>(ws);
    a.cl = cl->dev;
    const hipError_t e = ss::launch_absorb(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "absorb launch failed: %s", hipGetErrorString(e));
    idx->first_detail = frame_hi;
    return SS_OK;
  });
}

size_t ss_clusters_retrieve_workspace_bytes(const ss_clusters* cl) {
  if (!cl) return 0;
  ss::ClusterQueryPlan p{};
  p.Hk = cl->desc.n_kv_heads; p.D = cl->desc.head_dim; p.max_clusters = cl->desc.max_clusters;
  return ss::cluster_query_workspace(p, nullptr);
}

ss_status ss_clusters_retrieve(const ss_clusters* cl, const ss_index* idx, const void* const* queries,
                               int32_t n_q, int32_t k_clusters, void* ws, size_t ws_bytes, void* stream,
                               int64_t* cluster_ids, float* scores, int64_t* first_frame,
                               int64_t* last_frame, int32_t* n_out) {
  return guarded([&]() -> ss_status {
    if (!cl || !idx) return fail(SS_ERR_INVALID_ARGUMENT, "cluster set or index is NULL");
    const ss_index_desc& d = idx->desc;
    if (cl->desc.n_layers != d.n_layers || cl->desc.n_kv_heads != d.n_kv_heads || cl->desc.head_dim != d.head_dim)
      return fail(SS_ERR_INVALID_ARGUMENT, "cluster set and index shapes differ");
    if (n_q < 1 || n_q > 4096) return fail(SS_ERR_INVALID_ARGUMENT, "n_q %d outside 1..4096", n_q);
    if (k_clusters < 1 || k_clusters > ss::kMaxSelect)
      return fail(SS_ERR_UNSUPPORTED, "k_clusters %d outside 1..%d", k_clusters, ss::kMaxSelect);
    if (!queries || !queries[d.n_layers - 1]) return fail(SS_ERR_INVALID_ARGUMENT, "last-layer queries are NULL");
    if (!aligned(queries[d.n_layers - 1], 16)) return fail(SS_ERR_INVALID_ARGUMENT, "queries not 16-byte aligned");
    if (!cluster_ids || !scores || !first_frame || !last_frame || !n_out)
      return fail(SS_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
    ss::ClusterQueryPlan p{};
    p.L = d.n_layers; p.Hq = d.n_q_heads; p.Hk = d.n_kv_heads; p.G = p.Hq / p.Hk; p.D = d.head_dim;
    p.nq = n_q; p.k = k_clusters; p.max_clusters = cl->desc.max_clusters;
    p.q_last = static_cast<const uint16_t*>(queries[d.n_layers - 1]);
    p.cl = cl->dev;
    const size_t need = ss::cluster_query_workspace(p, nullptr);
    if (!ws || !aligned(ws, 256) || ws_bytes < need)
      return fail(SS_ERR_WORKSPACE, "cluster retrieval workspace NULL, misaligned or below %zu bytes", need);
    ss::cluster_query_workspace(p, ws);
    p.out_ids = cluster_ids; p.out_scores = scores; p.out_first = first_frame; p.out_last = last_frame;
    p.out_n = n_out;
    const hipError_t e = ss::launch_cluster_query(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "cluster retrieval launch failed: %s", hipGetErrorString(e));
    return SS_OK;
  });
}

ss_status ss_clusters_export(const ss_clusters* cl, int32_t* state, float* centroids, int32_t* sizes,
                             int64_t* span, float* reps, void* stream) {
  return guarded([&]() -> ss_status {
    if (!cl) return fail(SS_ERR_INVALID_ARGUMENT, "cluster set is NULL");
    const ss_cluster_desc& c = cl->desc;
    const size_t M = (size_t)c.max_clusters, dim = (size_t)c.n_kv_heads * c.head_dim;
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    struct Part { void* dst; const void* src; size_t bytes; } parts[] = {
        {state, cl->dev.state, 8},
        {centroids, cl->dev.centroids, M * dim * 4},
        {sizes, cl->dev.sizes, M * 4},
        {span, cl->dev.span, M * 16},
        {reps, cl->dev.reps, M * c.n_layers * dim * c.rows_per_unit * 4}};
    for (const Part& q : parts) {
      if (!q.dst) continue;
      const hipError_t e = hipMemcpyAsync(q.dst, q.src, q.bytes, hipMemcpyDeviceToDevice, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "cluster export: %s", hipGetErrorString(e));
    }
    return SS_OK;
  });
}

size_t ss_pooled_workspace_bytes(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                                  int32_t n_select) {
  if (check_pooled(idx, n_streams, n_q, n_select) != SS_OK) return 0;
  return pooled_ws(idx, n_streams, n_q, n_select);
}

ss_status ss_retrieve_pooled(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                             const int32_t* n_q, int32_t n_select, void* ws, size_t ws_bytes,
                             void* stream, int64_t* frame_ids, float* scores, int32_t* n_out) {
  return guarded([&]() -> ss_status {
    ss_status st = check_pooled(idx, n_streams, n_q, n_select);
    if (st) return st;
    if (!queries) return fail(SS_ERR_INVALID_ARGUMENT, "queries is NULL");
    const int L = idx[0]->desc.n_layers;
    for (int i = 0; i < n_streams * L; ++i) {
      if (!queries[i]) return fail(SS_ERR_INVALID_ARGUMENT, "queries[%d] is NULL", i);
      if (!aligned(queries[i], 16)) return fail(SS_ERR_INVALID_ARGUMENT, "queries[%d] not 16-byte aligned", i);
    }
    if (!frame_ids || !scores || !n_out) return fail(SS_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
    if (!ws || !aligned(ws, 256)) return fail(SS_ERR_WORKSPACE, "workspace NULL or not 256-byte aligned");
    const size_t need = pooled_ws(idx, n_streams, n_q, n_select);
    if (ws_bytes < need) return fail(SS_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", ws_bytes, need);
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    for (int s0 = 0; s0 < n_streams; s0 += ss::kMaxStreams) {
      ss::PooledPlan p;
      build_pooled(p, idx, s0, std::min(ss::kMaxStreams, n_streams - s0), queries, n_q, n_select);
      ss::pooled_workspace(p, ws);
      p.out_ids = frame_ids + (size_t)s0 * n_select;
      p.out_scores = scores + (size_t)s0 * n_select;
      p.out_n = n_out + s0;
      const hipError_t e = ss::launch_pooled(p, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "pooled ranking launch failed: %s", hipGetErrorString(e));
    }
    return SS_OK;
  });
}

int32_t ss_evidence_max_units(const ss_evidence_params* params, int32_t n_select, int32_t k_clusters) {
  const int64_t n = evidence_units_max(params, n_select, k_clusters);
  return (n < 0 || n > ss::kMaxEvidence) ? 0 : (int32_t)std::max<int64_t>(n, 1);
}

ss_status ss_assemble_evidence(ss_index* const* idx, int32_t n_streams, const int64_t* frame_ids,
                               int32_t n_select, const ss_evidence_clusters* clusters,
                               const ss_evidence_params* params, void* stream, int64_t* units, int32_t* kinds,
                               int32_t* n_units, int32_t max_units) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    if (n_streams < 1) return fail(SS_ERR_INVALID_ARGUMENT, "n_streams must be >= 1");
    for (int s = 0; s < n_streams; ++s)
      if (!idx[s]) return fail(SS_ERR_INVALID_ARGUMENT, "idx[%d] is NULL", s);
    const int kc = clusters ? clusters->k_clusters : 0;
    if (clusters && (kc < 1 || kc > ss::kMaxSelect))
      return fail(SS_ERR_UNSUPPORTED, "k_clusters %d outside 1..%d", kc, ss::kMaxSelect);
    const int64_t need = evidence_units_max(params, n_select, kc);
    if (need < 0) return fail(SS_ERR_INVALID_ARGUMENT, "invalid evidence parameters");
    if (need > ss::kMaxEvidence)
      return fail(SS_ERR_UNSUPPORTED, "%lld candidate items per stream > %d", (long long)need, ss::kMaxEvidence);
    if (max_units < std::max<int64_t>(need, 1) || max_units > ss::kMaxEvidence)
      return fail(SS_ERR_INVALID_ARGUMENT, "max_units %d outside %lld..%d", max_units,
                  (long long)std::max<int64_t>(need, 1), ss::kMaxEvidence);
    if (params->retrieved && !frame_ids) return fail(SS_ERR_INVALID_ARGUMENT, "frame_ids is NULL");
    if (!units || !n_units) return fail(SS_ERR_INVALID_ARGUMENT, "an output pointer is NULL");
    if (clusters && !kinds) return fail(SS_ERR_INVALID_ARGUMENT, "kinds is NULL (needed with clusters)");
    if (!aligned(units, 8) || !aligned(n_units, 4) || (kinds && !aligned(kinds, 4)) ||
        (frame_ids && !aligned(frame_ids, 8)))
      return fail(SS_ERR_INVALID_ARGUMENT, "misaligned device pointer");
    if (clusters) {
      if (!clusters->sets) return fail(SS_ERR_INVALID_ARGUMENT, "clusters->sets is NULL");
      if (params->retrieved && !clusters->cluster_ids)
        return fail(SS_ERR_INVALID_ARGUMENT, "clusters->cluster_ids is NULL");
      if (clusters->cluster_ids && !aligned(clusters->cluster_ids, 8))
        return fail(SS_ERR_INVALID_ARGUMENT, "misaligned device pointer");
      for (int s = 0; s < n_streams; ++s) {
        const ss_clusters* c = clusters->sets[s];
        if (c && (c->desc.n_layers != idx[s]->desc.n_layers || c->desc.n_kv_heads != idx[s]->desc.n_kv_heads ||
                  c->desc.head_dim != idx[s]->desc.head_dim))
          return fail(SS_ERR_INVALID_ARGUMENT, "cluster set %d and index %d shapes differ", s, s);
      }
    }
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    for (int s0 = 0; s0 < n_streams; s0 += ss::kMaxStreams) {
      ss::EvidenceArgs a{};
      a.S = std::min(ss::kMaxStreams, n_streams - s0);
      a.n_select = params->retrieved ? n_select : 0;
      a.n_recent = params->n_recent;
      a.n_before = params->n_before;
      a.n_after = params->n_after;
      a.retrieved = params->retrieved;
      a.max_units = max_units;
      for (int s = 0; s < a.S; ++s) {
        const ss_index* x = idx[s0 + s];
        a.T[s] = x->n_frames;
        a.lo[s] = std::min(x->first_detail, x->n_frames);
      }
      a.frame_ids = params->retrieved ? frame_ids + (size_t)s0 * n_select : nullptr;
      if (clusters && params->retrieved) {
        a.k_clusters = kc;
        a.cluster_ids = clusters->cluster_ids + (size_t)s0 * kc;
        for (int s = 0; s < a.S; ++s) {
          const ss_clusters* c = clusters->sets[s0 + s];
          a.cl_span[s] = c ? c->dev.span : nullptr;
          a.cl_count[s] = c ? c->dev.state : nullptr;
        }
      }
      a.units = units + (size_t)s0 * max_units;
      a.kinds = kinds ? kinds + (size_t)s0 * max_units : nullptr;
      a.n_units = n_units + s0;
      const hipError_t e = ss::launch_evidence(a, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "evidence launch failed: %s", hipGetErrorString(e));
    }
    return SS_OK;
  });
}

size_t ss_index_required_bytes(const ss_index_desc* desc) {
  if (check_desc(desc) != SS_OK) return 0;
  return layout(*desc).total;
}

ss_status ss_index_create(const ss_index_desc* desc, void* dev_arena, size_t arena_bytes,
                          ss_index** out) {
  return guarded([&]() -> ss_status {
    if (!out) return fail(SS_ERR_INVALID_ARGUMENT, "out is NULL");
    ss_status st = check_desc(desc);
    if (st) return st;
    if (!dev_arena) return fail(SS_ERR_INVALID_ARGUMENT, "arena is NULL");
    if (!aligned(dev_arena, 256)) return fail(SS_ERR_INVALID_ARGUMENT, "arena not 256-byte aligned");
    const Layout L = layout(*desc);
    if (arena_bytes < L.total)
      return fail(SS_ERR_CAPACITY, "arena %zu bytes, %zu needed", arena_bytes, L.total);
    ss_index* x = new (std::nothrow) ss_index();
    if (!x) return fail(SS_ERR_INTERNAL, "out of host memory");
    x->desc = *desc;
    x->arena = dev_arena;
    x->arena_bytes = arena_bytes;
    char* b = static_cast<char*>(dev_arena);
    x->dev.keys = reinterpret_cast<uint16_t*>(b + L.keys);
    x->dev.counts = reinterpret_cast<int32_t*>(b + L.counts);
    x->dev.desc = reinterpret_cast<float*>(b + L.desc);
    x->dev.pooled = reinterpret_cast<float*>(b + L.pooled);
    x->dev.stats = reinterpret_cast<uint32_t*>(b + L.stats);
    x->dev.frame_off = reinterpret_cast<int32_t*>(b + L.off);
    x->n_frames = 0;
    x->n_rows = 0;
    x->off.assign(1, 0);
    x->rpf = -1;
    *out = x;
    return SS_OK;
  });
}

ss_status ss_index_destroy(ss_index* idx) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    delete idx;
    return SS_OK;
  });
}

ss_status ss_index_info(const ss_index* idx, int64_t* n_frames, int64_t* n_rows) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    if (n_frames) *n_frames = idx->n_frames;
    if (n_rows) *n_rows = idx->n_rows;
    return SS_OK;
  });
}

ss_status ss_index_window(const ss_index* idx, int64_t* first_stored, int64_t* first_detail) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    if (first_stored) *first_stored = idx->frame_base;
    if (first_detail) *first_detail = idx->first_detail;
    return SS_OK;
  });
}

ss_status ss_index_compact(ss_index* idx, void* stream) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    const int64_t fs = idx->first_detail - idx->frame_base;
    if (fs <= 0) return SS_OK;
    const int64_t rs = row_of(idx, idx->first_detail);
    // the new host offsets first, so that nothing after the launch can fail
    std::vector<int64_t> off(idx->off.begin() + fs, idx->off.end());
    for (int64_t& v : off) v -= rs;
    ss::CompactArgs a{};
    const ss_index_desc& d = idx->desc;
    a.dev = idx->dev;
    a.L = d.n_layers; a.Hk = d.n_kv_heads; a.D = d.head_dim; a.max_rows = d.max_rows;
    a.row_shift = rs;
    a.keep_rows = idx->n_rows - rs;
    a.frame_shift = fs;
    a.keep_frames = idx->n_frames - idx->first_detail;
    const hipError_t e = ss::launch_compact(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "compaction launch failed: %s", hipGetErrorString(e));
    idx->off.swap(off);
    idx->frame_base = idx->first_detail;
    idx->n_rows = a.keep_rows;
    return SS_OK;
  });
}

ss_status ss_index_budget_split(const ss_index* idx, uint64_t budget_bytes, int64_t* frame_hi) {
  return guarded([&]() -> ss_status {
    if (!idx || !frame_hi) return fail(SS_ERR_INVALID_ARGUMENT, "idx or frame_hi is NULL");
    const ss_index_desc& d = idx->desc;
    const uint64_t L = (uint64_t)d.n_layers, Hk = (uint64_t)d.n_kv_heads, D = (uint64_t)d.head_dim;
    auto bytes = [&](int64_t f) {
      const uint64_t rows = (uint64_t)(row_of(idx, f + 1) - row_of(idx, f));
      return rows * L * Hk * (2 * D + 4) + (Hk * D + L * Hk * D) * 4 + 4;
    };
    const int64_t T = idx->n_frames, lo = idx->first_detail;
    const int64_t hi = std::max(lo, T - (int64_t)d.n_recent);   // the recent window stays detailed
    uint64_t mem = 0;
    for (int64_t f = lo; f < T; ++f) mem += bytes(f);
    int64_t h = lo;
    while (h < hi && mem > budget_bytes) mem -= bytes(h++);
    *frame_hi = h;
    return SS_OK;
  });
}

ss_status ss_index_append(ss_index* idx, const void* const* layer_keys, int32_t n_frames,
                          int32_t n_tokens, const ss_compress* compress, void* stream,
                          int64_t* first_frame_id) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    const ss_index_desc& d = idx->desc;
    if (!layer_keys) return fail(SS_ERR_INVALID_ARGUMENT, "layer_keys is NULL");
    if (n_frames < 1 || n_tokens < 1)
      return fail(SS_ERR_INVALID_ARGUMENT, "n_frames and n_tokens must be >= 1");
    if ((int64_t)n_frames * n_tokens > 0x7FFFFFFF)
      return fail(SS_ERR_UNSUPPORTED, "n_frames * n_tokens exceeds 2^31-1");
    for (int l = 0; l < d.n_layers; ++l) {
      if (!layer_keys[l]) return fail(SS_ERR_INVALID_ARGUMENT, "layer_keys[%d] is NULL", l);
      if (!aligned(layer_keys[l], 16))
        return fail(SS_ERR_INVALID_ARGUMENT, "layer_keys[%d] not 16-byte aligned", l);
    }
    int rpf = n_tokens;
    if (compress) {
      if (compress->n_centroids < 1 || compress->n_centroids > ss::kMaxCentroids)
        return fail(SS_ERR_UNSUPPORTED, "n_centroids %d outside 1..%d", compress->n_centroids,
                    ss::kMaxCentroids);
      if (compress->n_iters < 0 || compress->n_iters > 100)
        return fail(SS_ERR_INVALID_ARGUMENT, "n_iters %d outside 0..100", compress->n_iters);
      if (n_tokens > ss::kMaxTokensCompress)
        return fail(SS_ERR_UNSUPPORTED, "compression supports at most %d tokens per frame",
                    ss::kMaxTokensCompress);
      rpf = std::min(compress->n_centroids, n_tokens);
    }
    const int64_t stored = idx->n_frames - idx->frame_base;
    if (stored + n_frames > d.max_frames)
      return fail(SS_ERR_CAPACITY, "%lld stored frames + %d exceeds max_frames %lld", (long long)stored,
                  n_frames, (long long)d.max_frames);
    const int64_t new_rows = (int64_t)n_frames * rpf;
    if (idx->n_rows + new_rows > d.max_rows)
      return fail(SS_ERR_CAPACITY, "%lld rows + %lld exceeds max_rows %lld", (long long)idx->n_rows,
                  (long long)new_rows, (long long)d.max_rows);
    // the host offsets are reserved before anything is enqueued, so that the
    // bookkeeping after the launch cannot fail and leave the index behind the
    // device state
    idx->off.reserve(idx->off.size() + (size_t)n_frames);
    ss::AppendArgs a{};
    a.L = d.n_layers;
    a.Hk = d.n_kv_heads;
    a.D = d.head_dim;
    a.n_frames = n_frames;
    a.n_tokens = n_tokens;
    a.max_rows = d.max_rows;
    a.row0 = idx->n_rows;
    a.frame0 = stored;        // per-frame arena entries sit at id - frame_base
    a.rows_per_frame = rpf;
    a.n_centroids = compress ? compress->n_centroids : 0;
    a.n_iters = compress ? compress->n_iters : 0;
    for (int l = 0; l < d.n_layers; ++l) a.src[l] = static_cast<const uint16_t*>(layer_keys[l]);
    a.dst = idx->dev;
    hipError_t e = hipSuccess;
    if (idx->n_frames == 0)   // the key-magnitude statistic starts with the first append
      e = ss::launch_zero32(reinterpret_cast<int32_t*>(idx->dev.stats), 1, static_cast<hipStream_t>(stream));
    if (e == hipSuccess) e = ss::launch_append(a, compress != nullptr, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "append launch failed: %s", hipGetErrorString(e));
    if (first_frame_id) *first_frame_id = idx->n_frames;
    for (int f = 1; f <= n_frames; ++f) idx->off.push_back(idx->n_rows + (int64_t)f * rpf);   // reserved
    idx->n_frames += n_frames;
    idx->n_rows += new_rows;
    idx->rpf = (idx->rpf == -1 || idx->rpf == rpf) ? rpf : 0;
    return SS_OK;
  });
}

size_t ss_retrieve_workspace_bytes(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                                   const ss_retrieve_params* params) {
  if (check_batch(idx, n_streams, n_q, params) != SS_OK) return 0;
  return batch_ws(idx, n_streams, n_q, params);
}

ss_status ss_retrieve(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                      const int32_t* n_q, const ss_retrieve_params* params, void* ws,
                      size_t ws_bytes, void* stream, int64_t* frame_ids, int32_t* votes,
                      float* mass, int32_t* n_out) {
  return guarded([&]() -> ss_status {
    return retrieve_common(idx, n_streams, queries, n_q, params, ws, ws_bytes, stream, frame_ids,
                           votes, mass, n_out, nullptr);
  });
}

ss_status ss_retrieve_noalloc(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                              const int32_t* n_q, const ss_retrieve_params* params, void* stream,
                              int64_t* frame_ids, int32_t* votes, float* mass, int32_t* n_out) {
  return guarded([&]() -> ss_status {
    ss_status st = check_batch(idx, n_streams, n_q, params);
    if (st) return st;
    const size_t need = batch_ws(idx, n_streams, n_q, params);
    if (need > ss::kNoAllocBytes)
      return fail(SS_ERR_WORKSPACE,
                  "this batch needs a %zu-byte workspace, above the %zu bytes of the library-owned one: "
                  "call ss_retrieve with a caller workspace, or split the batch",
                  need, ss::kNoAllocBytes);
    void* ws = nullptr;
    const hipError_t e = ss::noalloc_workspace(&ws);
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "library workspace lookup failed: %s", hipGetErrorString(e));
    return retrieve_common(idx, n_streams, queries, n_q, params, ws, ss::kNoAllocBytes, stream, frame_ids,
                           votes, mass, n_out, nullptr);
  });
}

ss_status ss_retrieve_debug(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                            const int32_t* n_q, const ss_retrieve_params* params, void* ws,
                            size_t ws_bytes, void* stream, int64_t* frame_ids, int32_t* votes,
                            float* mass, int32_t* n_out, const ss_debug_out* dbg) {
  return guarded([&]() -> ss_status {
    if (!dbg) return fail(SS_ERR_INVALID_ARGUMENT, "dbg is NULL");
    return retrieve_common(idx, n_streams, queries, n_q, params, ws, ws_bytes, stream, frame_ids,
                           votes, mass, n_out, dbg);
  });
}

size_t ss_debug_scores_workspace_bytes(const ss_index* idx) {
  if (!idx) return 0;
  const ss_index_desc& d = idx->desc;
  return align256((size_t)d.n_layers * d.n_kv_heads * 2 * (d.head_dim / 32) * 64 * 16);
}

ss_status ss_debug_scores(const ss_index* idx, const void* const* queries, int32_t n_q,
                          int32_t layer, int32_t q_head, int32_t head_mode, int64_t row0,
                          int64_t n_rows, float* out, void* ws, size_t ws_bytes, void* stream) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    const ss_index_desc& d = idx->desc;
    if (!queries) return fail(SS_ERR_INVALID_ARGUMENT, "queries is NULL");
    for (int l = 0; l < d.n_layers; ++l)
      if (!queries[l] || !aligned(queries[l], 16))
        return fail(SS_ERR_INVALID_ARGUMENT, "queries[%d] NULL or not 16-byte aligned", l);
    if (n_q < 1 || n_q > 4096) return fail(SS_ERR_INVALID_ARGUMENT, "n_q %d outside 1..4096", n_q);
    if (head_mode != 0 && head_mode != 1) return fail(SS_ERR_INVALID_ARGUMENT, "head_mode must be 0 or 1");
    if (head_mode == 1 && d.n_kv_heads > 8)
      return fail(SS_ERR_UNSUPPORTED, "head_mode 1 supports at most 8 KV heads");
    if (layer < 0 || layer >= d.n_layers) return fail(SS_ERR_INVALID_ARGUMENT, "layer out of range");
    if (head_mode == 0 && (q_head < 0 || q_head >= d.n_q_heads))
      return fail(SS_ERR_INVALID_ARGUMENT, "q_head out of range");
    if (row0 < 0 || n_rows < 0 || row0 + n_rows > idx->n_rows)
      return fail(SS_ERR_INVALID_ARGUMENT, "rows [%lld, %lld) outside the %lld stored rows",
                  (long long)row0, (long long)(row0 + n_rows), (long long)idx->n_rows);
    if (!out && n_rows > 0) return fail(SS_ERR_INVALID_ARGUMENT, "out is NULL");
    if (!ws || !aligned(ws, 256) || ws_bytes < ss_debug_scores_workspace_bytes(idx))
      return fail(SS_ERR_WORKSPACE, "debug-scores workspace too small or misaligned");
    ss::RetrievePlan p;
    std::memset(&p, 0, sizeof p);
    p.S = 1;
    p.L = d.n_layers;
    p.Hq = d.n_q_heads;
    p.Hk = d.n_kv_heads;
    p.G = p.Hq / p.Hk;
    p.D = d.head_dim;
    p.head_mode = head_mode;
    p.NL = head_mode == 0 ? p.L * p.Hq : p.L;
    p.ncol = head_mode == 0 ? p.G : 1;
    p.ngs = head_mode == 0 ? p.Hk : 1;
    p.chunk_rows = kChunkRows;
    p.qB = static_cast<uint32_t*>(ws);
    ss::StreamPlan& sp = p.st[0];
    sp.keys = idx->dev.keys;
    sp.row_stride = (int32_t)d.max_rows;
    sp.nq = n_q;
    double sc = 1.0 / ((double)n_q * std::sqrt((double)p.D));
    if (head_mode == 1) sc /= (double)p.Hq;
    sp.qscale = (float)sc;
    for (int l = 0; l < p.L; ++l) sp.q[l] = static_cast<const uint16_t*>(queries[l]);
    const hipError_t e =
        ss::launch_debug_scores(p, layer, q_head, row0, n_rows, out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(SS_ERR_DEVICE, "debug scores launch failed: %s", hipGetErrorString(e));
    return SS_OK;
  });
}

ss_status ss_index_export(const ss_index* idx, void* rows_dev, int32_t* counts_dev, float* desc_dev,
                          int64_t* frame_offsets_host, void* stream) {
  return guarded([&]() -> ss_status {
    if (!idx) return fail(SS_ERR_INVALID_ARGUMENT, "idx is NULL");
    const ss_index_desc& d = idx->desc;
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    const size_t lg = (size_t)d.n_layers * d.n_kv_heads;
    if (frame_offsets_host)
      std::memcpy(frame_offsets_host, idx->off.data(), idx->off.size() * sizeof(int64_t));
    if (idx->n_rows > 0 && rows_dev) {
      const size_t rb = (size_t)idx->n_rows * d.head_dim * 2;
      const hipError_t e = hipMemcpy2DAsync(rows_dev, rb, idx->dev.keys, (size_t)d.max_rows * d.head_dim * 2,
                                            rb, lg, hipMemcpyDeviceToDevice, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "export rows: %s", hipGetErrorString(e));
    }
    if (idx->n_rows > 0 && counts_dev) {
      const size_t rb = (size_t)idx->n_rows * 4;
      const hipError_t e = hipMemcpy2DAsync(counts_dev, rb, idx->dev.counts, (size_t)d.max_rows * 4, rb, lg,
                                            hipMemcpyDeviceToDevice, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "export counts: %s", hipGetErrorString(e));
    }
    const int64_t stored = idx->n_frames - idx->frame_base;
    if (stored > 0 && desc_dev) {
      const hipError_t e = hipMemcpyAsync(desc_dev, idx->dev.desc,
                                          (size_t)stored * d.n_kv_heads * d.head_dim * 4,
                                          hipMemcpyDeviceToDevice, hs);
      if (e != hipSuccess) return fail(SS_ERR_DEVICE, "export descriptors: %s", hipGetErrorString(e));
    }
    return SS_OK;
  });
}

ss_status ss_debug_sample_plan(int64_t n_rows, int32_t top_k, int32_t* out) {
  return guarded([&]() -> ss_status {
    if (!out) return fail(SS_ERR_INVALID_ARGUMENT, "out is NULL");
    if (n_rows < 0 || n_rows > (int64_t)0x7FFFFFFF - 1)
      return fail(SS_ERR_INVALID_ARGUMENT, "n_rows %lld outside 0..2^31-2", (long long)n_rows);
    if (top_k < 1 || top_k > ss::kMaxTopK)
      return fail(SS_ERR_UNSUPPORTED, "top_k %d outside 1..%d", top_k, ss::kMaxTopK);
    const StreamSizes z = plan_stream(n_rows, 0, top_k);
    out[0] = z.m;
    out[1] = z.r;
    out[2] = (int32_t)candidate_cap(top_k, n_rows);
    out[3] = z.kk > 0 ? (int32_t)expected_candidates(n_rows, z.kk) : 0;
    return SS_OK;
  });
}

ss_status ss_set_profile_events(void* ev_start, void* ev_stop) {
  return guarded([&]() -> ss_status {
    if ((ev_start == nullptr) != (ev_stop == nullptr))
      return fail(SS_ERR_INVALID_ARGUMENT, "give both events or neither");
    g_ev_start = static_cast<hipEvent_t>(ev_start);
    g_ev_stop = static_cast<hipEvent_t>(ev_stop);
    return SS_OK;
  });
}

const char* ss_status_string(ss_status s) {
  switch (s) {
    case SS_OK: return "ok";
    case SS_ERR_INVALID_ARGUMENT: return "invalid argument";
    case SS_ERR_UNSUPPORTED: return "unsupported";
    case SS_ERR_CAPACITY: return "capacity exceeded";
    case SS_ERR_WORKSPACE: return "workspace too small";
    case SS_ERR_DEVICE: return "device error";
    case SS_ERR_INTERNAL: return "internal error";
    default: return "unknown status";
  }
}

const char* ss_last_error(void) { return g_err; }

int32_t ss_version(void) { return 1; }

}  // extern "C"
