// Internal declarations shared by the C-ABI layer (ss_api.cpp) and the gfx950
// kernels (ss_kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace ss {

// Streams handled by one launch of the retrieval pipeline (larger batches are
// split by the host into groups of this size).
constexpr int kMaxStreams = 32;
constexpr int kMaxGroup = 16;        // G = H_q / H_kv: one 16-column MFMA B tile
constexpr int kMaxTopK = 2048;
constexpr int kMaxSelect = 64;
constexpr int kMaxPool = 256;
constexpr int kTile = 16;            // key rows per MFMA tile
constexpr int kMaxTokensCompress = 256;
constexpr int kMaxCentroids = 64;
constexpr int kMaxLayers = 32;
constexpr int kMaxListsPerStream = 4096;  // n_layers * n_q_heads

// The host-side RetrievePlan is never passed to a kernel as a whole; each
// kernel receives a compact argument struct built from it.

// Device view of one index arena.
struct IndexDev {
  uint16_t* keys;       // [L][H_kv][max_rows][d] bf16
  int32_t* counts;      // [L][H_kv][max_rows]
  float* desc;          // [max_frames][H_kv*d]
  float* pooled;        // [max_frames][L][H_kv][d] mean raw key per (frame, layer, KV head)
  int32_t* frame_off;   // [max_frames+1]
  uint32_t* stats;      // [0]: the largest |raw key element| appended so far (float bits)
};

// ---------------------------------------------------------------------------
// Append
// ---------------------------------------------------------------------------
struct AppendArgs {
  int L, Hk, D;
  int n_frames, n_tokens;
  int64_t max_rows;
  int64_t row0;          // first destination row
  int64_t frame0;        // first new frame id
  int rows_per_frame;    // n_tokens raw, min(n_centroids, n_tokens) compressed
  int n_centroids, n_iters;
  const uint16_t* src[kMaxLayers];  // per layer [H_kv][n_frames*n_tokens][d]
  IndexDev dst;
};

hipError_t launch_append(const AppendArgs& a, bool compress, hipStream_t st);

// ---------------------------------------------------------------------------
// Retrieval
// ---------------------------------------------------------------------------
struct StreamPlan {
  const uint16_t* keys;
  const int32_t* frame_off;
  const float* desc;
  int32_t row_stride;    // max_rows of the index
  int32_t n;             // candidate rows
  int32_t f;             // candidate frames
  int32_t m;             // sampled rows
  int32_t r;             // rank of the sample threshold
  int32_t kk;            // min(top_k, n)
  int32_t nq;
  int32_t rpf;           // rows per frame when every frame has the same count, else 0
  int64_t frame0;        // first candidate frame (earlier ones are in long-term clusters)
  int64_t hist0;         // its place among the frames the arena stores (frame0 - the first stored frame)
  int64_t row0;          // its first row; keys, frame_off and desc above start there
  const uint32_t* kmax;  // the index's largest |key element| (float bits, device)
  float qscale;          // 1 / (n_q sqrt(d)) (head_mode 0), further / H_q (head_mode 1)
  const uint16_t* q[kMaxLayers];  // per layer query pointer [H_q][n_q][d]
};

struct RetrievePlan {
  int S, L, Hq, Hk, G, D;
  int head_mode;
  int score_mode;        // 0 scaled logits, 1 attention probabilities
  bool hm_prob;          // head_mode 1 with attention probabilities: per-head scores throughout
  int NL;                // lists per stream
  int NLs;               // sampled lists per stream: NL, or L * H_q when hm_prob (one per head)
  int ncol;              // MFMA output columns used per item (G or 1)
  int ngs;               // KV-head sets per layer: H_kv (head_mode 0) or 1
  int top_k, n_select, pool, pool_mult;
  int cap;               // candidate capacity per list
  int k_max;             // max over streams of kk
  int m_max, f_max;
  int chunk_rows, samp_chunk;
  StreamPlan st[kMaxStreams];

  // workspace carve (device pointers)
  uint32_t* qB;          // [S][L][H_kv][2][d/32][64] uint4
  uint32_t* tau;         // [S*NL]
  uint32_t* cnt;         // [S*NL]
  float* samp;           // [S*NLs][m_max]
  uint64_t* below;       // score_mode 1: fixed-point sums of exp over the rows below each cut-off,
                         // [S*NL] (head mode 0) or [S*L*H_q] (hm_prob)
  float* lhat;           // hm_prob: [S*L*H_q] sample estimates of each head's log-sum-exp
  float* cand_sc;        // hm_prob: [S*NL][H_q][cap] per-head logits of the candidates
  uint32_t* left_max;    // hm_prob: [S*NL] largest estimate among the rows the streaming pass left out
  float* alpha;          // hm_prob: [S*NL][m_max] estimated attention of the sampled rows
  float* cand_lse;       // hm_prob: [S*NL][H_q] exact log-sum-exp of each head's list
  uint64_t* cand;        // [S*NL][cap]
  float* qcol;           // [S][L][H_kv][16] L1 norms of the scaled query columns
  int32_t* sexp;         // [S] fixed-point exponent of each stream's attention mass
  uint32_t* dyn_ctr;     // chunk counters of the streaming pass
  int32_t* votes;        // [S][f_max] per-frame votes
  int64_t* massfx;       // [S][f_max] per-frame mass at scale 2^sexp
  uint64_t* rec_hi;      // [S][f_max] compacted (votes, mass, frame) records
  uint64_t* rec_lo;
  int32_t* pool_ids;     // [S][pool]
  int32_t* pool_votes;   // [S][pool]
  float* pool_mass;      // [S][pool]
  int32_t* pool_n;       // [S]
  float* gram;           // [S][pool][pool]

  // outputs
  int64_t* out_ids;
  int32_t* out_votes;
  float* out_mass;
  int32_t* out_n;
  int out_stride;        // n_select

  // optional debug outputs
  int32_t* dbg_topk_pos;
  float* dbg_topk_score;
  int32_t* dbg_vote_hist;
  float* dbg_mass_hist;
  int32_t* dbg_pool;
  int32_t* dbg_pool_n;
  int32_t* dbg_list_stats;
  int dbg_hist_stride;   // largest max_frames of the batch

  // profiling hook around the streaming kernel
  hipEvent_t ev_start, ev_stop;
};

// Bytes of each workspace region for a plan; fills the plan's pointers when
// `ws` is non-null.  Returns the total.
size_t carve_workspace(RetrievePlan& p, void* ws);

hipError_t launch_retrieve(RetrievePlan& p, hipStream_t st);

// The library-owned retrieval workspace of the no-alloc entry point: a
// file-scope device array of kNoAllocBytes on every device the library runs
// on.  noalloc_workspace() returns its device address on the current device
// (looked up once per device with hipGetSymbolAddress).
constexpr size_t kNoAllocBytes = (size_t)64 << 20;
hipError_t noalloc_workspace(void** ptr);

// Pooled shallow Q-K ranking of up to kMaxStreams streams.
struct PooledPlan {
  int S, L, Hq, Hk, G, D, n_select;
  int64_t F[kMaxStreams];               // candidate frames per stream
  int64_t frame0[kMaxStreams];          // id of the first candidate frame
  const float* pooled[kMaxStreams];     // per stream, from the first candidate frame: [F][L][H_kv][d]
  const uint16_t* q[kMaxStreams * kMaxLayers];  // [s * L + l] -> bf16 [H_q][n_q][d]
  int32_t nq[kMaxStreams];
  int64_t f_max;
  float* w;        // workspace [S][L][H_kv][d]: pooled query weights
  float* scores;   // workspace [S][f_max]
  int64_t* out_ids;
  float* out_scores;
  int32_t* out_n;
};
size_t pooled_workspace(PooledPlan& p, void* ws);   // fills p.w / p.scores when ws != null
hipError_t launch_pooled(const PooledPlan& p, hipStream_t st);

// Long-term clusters of one stream (device view of a cluster arena).
struct ClusterDev {
  int32_t* state;      // [0] clusters in use, [1] 1 once a unit had to join a full set
  float* centroids;    // [max_clusters][H_kv*d]
  int32_t* sizes;      // [max_clusters]
  int64_t* span;       // [max_clusters][2]: first and last member frame
  float* reps;         // [max_clusters][L][H_kv][rows][d]: running-average keys
};

struct AbsorbArgs {
  int L, Hk, D, R;            // R: stored rows of every absorbed unit
  int64_t max_clusters, max_rows;
  float tau;
  int64_t f_lo;               // first leaving frame
  int n_units;
  int64_t row_lo;             // its first row
  const float* desc;          // descriptors of the leaving frames [n_units][H_kv*d]
  const uint16_t* keys;       // index keys [L][H_kv][max_rows][d]
  int32_t* assign;            // workspace [n_units][2]: cluster, members before joining
  ClusterDev cl;
};
hipError_t launch_absorb(const AbsorbArgs& a, hipStream_t st);
hipError_t launch_zero32(int32_t* p, int n, hipStream_t st);   // a kernel, not a memset node

struct ClusterQueryPlan {
  int L, Hq, Hk, G, D, nq, k;
  const uint16_t* q_last;     // last shallow layer's queries [H_q][n_q][d]
  int64_t max_clusters;
  ClusterDev cl;
  float* w;                   // workspace [H_kv*d]
  float* scores;              // workspace [max_clusters]
  int64_t* out_ids;
  float* out_scores;
  int64_t* out_first;
  int64_t* out_last;
  int32_t* out_n;
};
size_t cluster_query_workspace(ClusterQueryPlan& p, void* ws);
hipError_t launch_cluster_query(const ClusterQueryPlan& p, hipStream_t st);

// Evidence assembly of up to kMaxStreams streams, one block each.
constexpr int kMaxEvidence = 4096;   // candidate units per stream (sorted in LDS)
struct EvidenceArgs {
  int S, n_select, n_recent, n_before, n_after, retrieved, max_units;
  int64_t T[kMaxStreams];        // frames stored per stream
  int64_t lo[kMaxStreams];       // first frame of each stream's detailed window
  const int64_t* frame_ids;      // [S][n_select], may be null when !retrieved
  // retrieved long-term clusters (k_clusters == 0: none)
  int k_clusters;
  const int64_t* cluster_ids;        // [S][k_clusters], -1 padded
  const int64_t* cl_span[kMaxStreams];   // per stream [max_clusters][2], null: no cluster set
  const int32_t* cl_count[kMaxStreams];  // per stream: clusters in use (device)
  int64_t* units;                // [S][max_units]
  int32_t* kinds;                // [S][max_units] 0 unit, 1 cluster, -1 padding; may be null
  int32_t* n_units;              // [S]
};
hipError_t launch_evidence(const EvidenceArgs& a, hipStream_t st);

// Compaction of an index arena: the stored frames from the first detailed one
// on move to the arena's start.  Rows [row_shift, row_shift + keep_rows) of
// every (layer, KV head) go to [0, keep_rows); the per-frame entries of the
// stored frames [frame_shift, frame_shift + keep_frames) go to [0,
// keep_frames), and the row offsets (keep_frames + 1 of them) are rebased by
// row_shift.
struct CompactArgs {
  IndexDev dev;
  int L, Hk, D;
  int64_t max_rows;
  int64_t row_shift, keep_rows;
  int64_t frame_shift, keep_frames;
};
hipError_t launch_compact(const CompactArgs& a, hipStream_t st);

// Scores of one list over a row range, same arithmetic as the retrieval.
hipError_t launch_debug_scores(RetrievePlan& p, int layer, int q_head, int64_t row0,
                               int64_t n_rows, float* out, hipStream_t st);

}  // namespace ss
