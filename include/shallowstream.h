/*
 * shallowstream.h -- C ABI of the MI355X (gfx950) library for ShallowStream's
 * query-time evidence retrieval over a shallow-layer key index.
 *
 * The method (Sec. 4 of the ShallowStream paper):
 *   - index construction (Sec. 4.1): every video unit ("frame") contributes the
 *     keys of its visual tokens at each shallow layer (Eq. shallow_streaming_cache)
 *     and a unit descriptor (Eq. memory_key); an optional per-frame k-means
 *     compression stores centroids instead of the raw token keys;
 *   - retrieval (Sec. 4.2, "Optional Evidence Retrieval"): scaled Q-K scores of
 *     the question against every stored key, top-k per list
 *     (Eq. token_vote_candidates), one vote per selected token for its frame,
 *     a vote-ranked pool of pool_mult*K frames (ties by attention mass) and
 *     greedy max-min diversity in descriptor space (DivTopK, Eq. selected_evidence).
 *
 * Conventions for every entry point:
 *   - bf16 arrays are raw IEEE bfloat16 bit patterns (uint16), row-major.
 *   - "device pointer" means memory of the current HIP device; "host pointer"
 *     means ordinary CPU memory.  `stream` is a hipStream_t (NULL = the
 *     default stream).  Work is enqueued on `stream`; the call returns without
 *     waiting for it.  Inputs must stay valid until that work completes.
 *   - The library never allocates device memory: the caller provides the index
 *     arena and every workspace and output buffer.
 *   - Every argument is validated on the host before anything is enqueued.  On
 *     failure the call returns a non-zero status, ss_last_error() describes it,
 *     and the index is unchanged.  No exception crosses this boundary.
 *   - Device faults surface at the caller's next synchronisation.
 *   - Calls on different indices may run concurrently.  Appends and retrievals
 *     touching one index must be ordered on one stream (or synchronised).
 *   - Inputs must be finite; NaN or Inf keys or queries give unspecified ranks.
 */
#ifndef SHALLOWSTREAM_H
#define SHALLOWSTREAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ss_index ss_index; /* opaque, host-side handle */
typedef int32_t ss_status;

enum {
  SS_OK = 0,
  SS_ERR_INVALID_ARGUMENT = 1, /* a pointer, shape or parameter is wrong        */
  SS_ERR_UNSUPPORTED = 2,      /* valid but outside what the kernels implement  */
  SS_ERR_CAPACITY = 3,         /* the arena cannot hold the appended frames     */
  SS_ERR_WORKSPACE = 4,        /* the workspace is smaller than required        */
  SS_ERR_DEVICE = 5,           /* a HIP runtime call or kernel launch failed    */
  SS_ERR_INTERNAL = 6
};

/* Shape and capacity of one stream's index.
 *   n_layers    L_s, the shallow layers kept (the pruning boundary P).
 *   n_q_heads   H_q query heads; n_kv_heads H_kv key heads, H_q % H_kv == 0,
 *               G = H_q / H_kv <= 16.  Query head h reads KV head h / G.
 *   head_dim    d, 64 or 128.
 *   max_frames  frame capacity; max_rows row capacity per (layer, KV head),
 *               with max_rows * head_dim * 2 < 2^31 (one (layer, KV head) of
 *               keys below 2 GiB: 8,388,607 rows at d = 128).
 *   n_recent    N_r: the newest n_recent frames are never retrieval
 *               candidates (Eq. context_partition); 0 makes every frame one. */
typedef struct {
  int32_t n_layers;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int64_t max_frames;
  int64_t max_rows;
  int32_t n_recent;
} ss_index_desc;

/* Per-frame k-means compression at append: each frame's tokens, per (layer,
 * KV head), become min(n_centroids, n_tokens) centroids: farthest-point
 * initialisation (first centre = the token farthest from the frame mean), then
 * exactly n_iters Lloyd rounds on squared Euclidean distance in fp32, ties to the
 * lower index, empty clusters keep their centre; stored as bf16 (nearest-even)
 * in farthest-point order.  1 <= n_centroids <= 64, 0 <= n_iters <= 100,
 * n_tokens <= 256. */
typedef struct {
  int32_t n_centroids;
  int32_t n_iters;
} ss_compress;

/* Retrieval parameters.
 *   top_k      k rows kept per list (Eq. token_vote_candidates), 1..2048; more
 *              than the candidate rows selects them all.
 *   n_select   K, the frame budget, 1..64.
 *   pool_mult  the vote-ranked pool holds pool_mult*K frames (4 in the paper),
 *              pool_mult*K <= 256; 1 makes diversity selection a no-op.
 *   head_mode  0: one list per (layer, query head).  1: one list per layer with
 *              the values averaged over all query heads (Sec. 4.2 averages the
 *              attention over heads).
 *   score_mode the value of a candidate row in a list.  0: the scaled logit
 *              q.k/sqrt(d) (mean over query tokens).  1: the Q-K attention
 *              probability, the softmax of one (layer, query head)'s logits
 *              over all candidate rows, so a head-mode-1 list averages
 *              per-head probabilities.  The attention mass of a frame is the
 *              sum of its selected rows' values.  In head mode 0 the lists and
 *              votes are the same in both modes (only the mass differs); in
 *              head mode 1 they differ.  Head mode 1 with score_mode 1 needs
 *              n_kv_heads in {1, 2, 4, 8} and n_kv_heads * head_dim <= 512.
 */
typedef struct {
  int32_t top_k;
  int32_t n_select;
  int32_t pool_mult;
  int32_t head_mode;
  int32_t score_mode;
} ss_retrieve_params;

/* Device bytes an index with this shape needs (0 if `desc` is invalid).
 * Layout (each part 256-byte aligned): keys bf16 [L_s][H_kv][max_rows][d];
 * member counts int32 [L_s][H_kv][max_rows]; descriptors fp32
 * [max_frames][H_kv*d]; pooled keys fp32 [max_frames][L_s][H_kv][d] (each
 * frame's mean raw key per layer and KV head); frame row offsets int32
 * [max_frames+1]; a 16-byte statistics block (the largest raw key magnitude
 * appended, which bounds every score and so fixes the fixed-point scale of
 * the attention mass). */
size_t ss_index_required_bytes(const ss_index_desc* desc);

/* Create an empty index over a caller-owned device arena of at least
 * ss_index_required_bytes(desc) bytes, 256-byte aligned: the full-history
 * shallow cache of Sec. 4.1 ("Full-History Shallow Cache", Eq.
 * shallow_streaming_cache) for L_s = P shallow layers, with room for each
 * unit's descriptor (Eq. memory_key).  Only keys are kept: the values of the
 * cache are not read by retrieval.  The arena must stay allocated until
 * ss_index_destroy; the library writes it only through ss_index_append.
 * *out receives the handle (host memory owned by the library).  Errors:
 * SS_ERR_INVALID_ARGUMENT / SS_ERR_UNSUPPORTED for a bad shape, SS_ERR_CAPACITY
 * when arena_bytes is too small; nothing is created then. */
ss_status ss_index_create(const ss_index_desc* desc, void* dev_arena, size_t arena_bytes,
                          ss_index** out);

/* Release the host-side handle.  The arena stays the caller's. */
ss_status ss_index_destroy(ss_index* idx);

/* Host-side counters: frames appended so far (frame ids run 0 .. n_frames-1)
 * and rows per (layer, KV head) the arena holds now. */
ss_status ss_index_info(const ss_index* idx, int64_t* n_frames, int64_t* n_rows);

/* The frames the index holds: the arena stores frames [first_stored,
 * n_frames) (frames below were dropped by ss_index_compact), and frames below
 * first_detail have left the detailed window for long-term clusters
 * (ss_clusters_absorb); first_stored <= first_detail.  Either pointer may be
 * NULL. */
ss_status ss_index_window(const ss_index* idx, int64_t* first_stored, int64_t* first_detail);

/* The memory side of long-history compression (Eq.
 * optional_context_compression): the frames that left the detailed window
 * leave the arena too.  Their rows, member counts, descriptors, pooled keys and
 * row offsets are dropped; the stored rows of the detailed frames move to the
 * start of every (layer, KV head) run of the arena (in passes of at most the
 * dropped rows, each a copy kernel on `stream`), so that later appends reuse
 * the space: max_frames and max_rows then bound the frames and rows kept in
 * detail, not the stream's length.  Frame ids stay as they were.  Retrieval,
 * pooled ranking, absorption and evidence are unchanged by it.  No-op when no
 * frame has left the detailed window since the last compaction.  Its cost is a
 * copy of the kept rows, so compact after absorbing many frames at once.
 * Ordered on `stream` with the index's other work like an append; on
 * SS_ERR_DEVICE the index must be discarded. */
ss_status ss_index_compact(ss_index* idx, void* stream);

/* Where the detailed window must start to fit a byte budget B (Eq.
 * optional_context_compression: once Mem(M_T) > B, older history leaves for
 * long-term clusters while the recent units and the near history stay in
 * detail).  Mem counts the arena bytes of the frames in the detailed window:
 * a frame of r stored rows takes r*L_s*H_kv*(2d + 4) + (1 + L_s)*H_kv*d*4 + 4
 * bytes (keys, member counts, descriptor, pooled keys, row offset).
 * *frame_hi (host) receives the smallest frame_hi in [first_detail,
 * max(first_detail, n_frames - n_recent)] whose frames [frame_hi, n_frames) fit
 * in budget_bytes, or the end of that range when none does (the recent window
 * always stays detailed); first_detail when the window already fits.  Pass it
 * to ss_clusters_absorb, then ss_index_compact.  Host work only. */
ss_status ss_index_budget_split(const ss_index* idx, uint64_t budget_bytes, int64_t* frame_hi);

/* Append n_frames frames of n_tokens visual tokens each: each unit's keys at
 * every shallow layer join the cache in temporal order (Sec. 4.1, Eq.
 * shallow_streaming_cache; frame t of the paper's stream is frame id t - 1
 * here), and its descriptor (Eq. memory_key) is computed on the device.
 *   layer_keys  host array of L_s device pointers; pointer l addresses bf16
 *               [H_kv][n_frames*n_tokens][d] keys of shallow layer l (16-byte
 *               aligned).  Frame f owns tokens [f*n_tokens, (f+1)*n_tokens).
 *   compress    NULL stores the raw keys; otherwise see ss_compress.
 *   first_frame_id  host out: the id of the first appended frame (frame ids are
 *               append order from 0).
 * The unit descriptor (Eq. memory_key) always uses the raw keys of the last
 * shallow layer.  Fails with SS_ERR_CAPACITY (index unchanged) if the frames or
 * rows do not fit; the host bookkeeping is reserved before any work is
 * enqueued, so an error return never leaves work behind on `stream`.  The
 * keys are read by the enqueued kernels: keep them valid until they finish. */
ss_status ss_index_append(ss_index* idx, const void* const* layer_keys, int32_t n_frames,
                          int32_t n_tokens, const ss_compress* compress, void* stream,
                          int64_t* first_frame_id);

/* Workspace bytes ss_retrieve needs for this batch in the indices' current state
 * (0 if the arguments are invalid).  n_q: host array of n_streams token counts. */
size_t ss_retrieve_workspace_bytes(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                                   const ss_retrieve_params* params);

/* Evidence retrieval for n_streams independent streams with one question each
 * (Sec. 4.2, "Optional Evidence Retrieval"): the candidate tokens are those of
 * every frame except the newest n_recent (Eq. context_partition) and, after
 * long-history compression, those of the detailed window only; each list
 * keeps its top_k tokens (Eq. token_vote_candidates), every selected token
 * votes for its frame, the pool_mult*n_select frames with the most votes
 * (ties by attention mass, then the lower frame id) form the pool, and greedy
 * max-min diversity over the descriptors of Eq. memory_key picks n_select of
 * them (DivTopK of Eq. selected_evidence).
 *   idx        host array of n_streams handles with identical shapes.
 *   queries    host array of n_streams*L_s device pointers, stream-major;
 *              pointer [s*L_s + l] addresses bf16 [H_q][n_q[s]][d] query states
 *              of layer l (post-RoPE, as cached; 16-byte aligned).  The score of
 *              a key is the mean over query tokens of the scaled logit
 *              q.k/sqrt(d) (the paper uses the last prompt token: n_q = 1).
 *   n_q        host array, per stream, 1..4096.
 *   ws         device workspace of ws_bytes >= ss_retrieve_workspace_bytes().
 * Outputs (device, [n_streams][n_select] each, selection order):
 *   frame_ids  int64 frame ids, -1 after the n_out[s] selected frames;
 *   votes      int32 votes of each selected frame (0 in the padding);
 *   mass       fp32 attention mass (sum of the frame's selected scores);
 *   n_out      int32 [n_streams], number of frames selected. */
ss_status ss_retrieve(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                      const int32_t* n_q, const ss_retrieve_params* params, void* ws,
                      size_t ws_bytes, void* stream, int64_t* frame_ids, int32_t* votes,
                      float* mass, int32_t* n_out);

/* ss_retrieve for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * workspace is a library-owned device buffer of SS_NOALLOC_WORKSPACE_BYTES
 * (64 MiB) on each device, which the runtime places when the library's code is
 * loaded on that device and keeps until the process ends; its address is
 * looked up on the first such call on a device.  The call allocates nothing
 * and frees nothing.  Arguments and outputs as in ss_retrieve, without ws.
 * Fails with SS_ERR_WORKSPACE, before enqueueing anything, when
 * ss_retrieve_workspace_bytes() of the batch exceeds SS_NOALLOC_WORKSPACE_BYTES
 * (a single one-hour stream of the 28/4-head, d = 128 shape needs about 10 MB;
 * a batch of 16 such streams does not fit).  Every call on one device shares
 * that buffer and leaves its contents behind (each call initialises what it
 * reads): calls that overlap on one device (unordered streams, or several host
 * threads) race and give undefined results, so order them on one stream. */
#define SS_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
ss_status ss_retrieve_noalloc(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                              const int32_t* n_q, const ss_retrieve_params* params, void* stream,
                              int64_t* frame_ids, int32_t* votes, float* mass, int32_t* n_out);

/* Intermediates of one retrieval, for parity checks (any pointer may be NULL).
 * Device arrays, n_lists = L_s*H_q (head_mode 0) or L_s (head_mode 1), lists
 * ordered layer-major, F = frames of the stream at the call:
 *   topk_pos    int32 [n_streams][n_lists][top_k] row positions in rank order
 *               (score desc, position asc), -1 padded;
 *   topk_score  fp32  same shape, the scores;
 *   vote_hist   int32 [n_streams][max_frames] votes of every stored frame,
 *               at frame id - first_stored (ss_index_window);
 *   mass_hist   fp32  [n_streams][max_frames] attention mass, likewise;
 *   pool        int32 [n_streams][pool_mult*n_select] the vote-ranked pool, -1 padded;
 *   pool_n      int32 [n_streams];
 *   list_stats  int32 [n_streams][n_lists][2]: candidates kept by the streaming
 *               pass, and 1 if the list took the exact fallback path. */
typedef struct {
  int32_t* topk_pos;
  float* topk_score;
  int32_t* vote_hist;
  float* mass_hist;
  int32_t* pool;
  int32_t* pool_n;
  int32_t* list_stats;
} ss_debug_out;

/* ss_retrieve plus the intermediates in `dbg`. */
ss_status ss_retrieve_debug(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                            const int32_t* n_q, const ss_retrieve_params* params, void* ws,
                            size_t ws_bytes, void* stream, int64_t* frame_ids, int32_t* votes,
                            float* mass, int32_t* n_out, const ss_debug_out* dbg);

/* Pooled shallow Q-K ranking, the baseline ranker of the paper's evidence-
 * ranker ablation: each candidate frame (all but the newest n_recent) is
 * scored by the mean over shallow layers l and query heads h of
 * qbar_{l,h} . Kbar_{l,h/G,t} / sqrt(d), where qbar is the mean query over the
 * question's tokens and Kbar the frame's mean raw key of that layer and KV head
 * (kept at append); for raw frames this is the mean of the frame's token
 * scores.  The n_select best frames by (score desc, frame asc) are returned,
 * with no diversity selection.  Arguments as in ss_retrieve; outputs (device,
 * [n_streams][n_select]): frame_ids int64 (-1 padded), scores fp32 (0 in the
 * padding), n_out int32 [n_streams].  n_select is 1..64. */
size_t ss_pooled_workspace_bytes(ss_index* const* idx, int32_t n_streams, const int32_t* n_q,
                                 int32_t n_select);
ss_status ss_retrieve_pooled(ss_index* const* idx, int32_t n_streams, const void* const* queries,
                             const int32_t* n_q, int32_t n_select, void* ws, size_t ws_bytes,
                             void* stream, int64_t* frame_ids, float* scores, int32_t* n_out);

/* Long-history compression (Sec. 4.1, "Optional Long-History Compression").
 * When the history outgrows its budget, the oldest detailed frames leave the
 * detailed window in temporal order (ss_clusters_absorb).  A leaving frame
 * joins the latest long-term cluster if its descriptor (Eq. memory_key) has
 * dot product >= tau with the cluster centroid, which becomes
 * Norm((n c + k) / (n + 1)); otherwise it starts a new cluster (Eq.
 * optional_long_memory_clustering).  Each cluster keeps the running average of
 * its members' stored key rows, position by position, at every shallow layer
 * (Eq. optional_long_memory_representative).  Frames that left the detailed
 * window are no longer token candidates for ss_retrieve / ss_retrieve_pooled
 * (their rows stay in the index arena); their clusters are ranked against the
 * question by ss_clusters_retrieve (Eq. selected_cluster_evidence).
 *   n_layers, n_kv_heads, head_dim   as the index's;
 *   rows_per_unit  stored rows of every absorbed frame (tokens, or centroids);
 *   max_clusters   capacity; a frame that would open a cluster beyond it joins
 *                  the latest cluster instead and sets the overflow flag;
 *   tau            the joining threshold (the paper gives no value). */
typedef struct {
  int32_t n_layers;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t rows_per_unit;
  int64_t max_clusters;
  float tau;
} ss_cluster_desc;

typedef struct ss_clusters ss_clusters;

/* Device bytes a cluster set needs (0 if `desc` is invalid).  Layout (256-byte
 * aligned parts): state int32 [2] (clusters in use, overflow flag); centroids
 * fp32 [max_clusters][n_kv_heads*head_dim]; sizes int32 [max_clusters];
 * member frame span int64 [max_clusters][2]; representatives fp32
 * [max_clusters][n_layers][n_kv_heads][rows_per_unit][head_dim]. */
size_t ss_clusters_required_bytes(const ss_cluster_desc* desc);

/* An empty cluster set over a caller-owned device arena (256-byte aligned, at
 * least ss_clusters_required_bytes); enqueues the zeroing of its state on
 * `stream`. */
ss_status ss_clusters_create(const ss_cluster_desc* desc, void* dev_arena, size_t arena_bytes,
                             void* stream, ss_clusters** out);
ss_status ss_clusters_destroy(ss_clusters* cl);

/* Frames [first, frame_hi) of `idx` leave its detailed window, in order, and
 * are folded into `cl`; `first` is where the previous call stopped (0 at the
 * start).  frame_hi must not reach into the recent window (the newest n_recent
 * frames), and every absorbed frame must store rows_per_unit rows.  ws: device
 * workspace of ss_clusters_absorb_workspace_bytes(frame_hi - first) bytes. */
size_t ss_clusters_absorb_workspace_bytes(int64_t n_frames);
ss_status ss_clusters_absorb(ss_clusters* cl, ss_index* idx, int64_t frame_hi, void* ws, size_t ws_bytes,
                             void* stream);

/* The k_clusters best clusters for one question (Eq. selected_cluster_evidence):
 * a centroid's score is the scaled logit of the mean query of the last shallow
 * layer against it, query head h meeting the centroid's block of KV head h/G,
 * averaged over query heads.  Ties go to the older cluster.  queries: host
 * array of n_layers device pointers as in ss_retrieve (only the last layer is
 * read).  Outputs (device, [k_clusters], rank order, -1 / 0 padded):
 * cluster_ids int64, scores fp32, first_frame and last_frame int64 member
 * span; n_out int32 [1].  k_clusters is 1..64. */
size_t ss_clusters_retrieve_workspace_bytes(const ss_clusters* cl);
ss_status ss_clusters_retrieve(const ss_clusters* cl, const ss_index* idx, const void* const* queries,
                               int32_t n_q, int32_t k_clusters, void* ws, size_t ws_bytes, void* stream,
                               int64_t* cluster_ids, float* scores, int64_t* first_frame,
                               int64_t* last_frame, int32_t* n_out);

/* Copy a cluster set out (parity only; device pointers, any may be NULL):
 * state int32 [2], centroids, sizes, span, representatives as laid out in
 * ss_clusters_required_bytes, for all max_clusters slots. */
ss_status ss_clusters_export(const ss_clusters* cl, int32_t* state, float* centroids, int32_t* sizes,
                             int64_t* span, float* reps, void* stream);

/* Evidence assembly parameters (Eq. selected_evidence).
 *   n_recent   N_r, the newest frames that are always evidence (Eq.
 *              context_partition); the paper uses 6 with retrieval, 2 without.
 *   n_before   frames before each selected frame added as its temporal
 *              neighbours (the paper: 1); n_after likewise after it (0).
 *   retrieved  the gate's decision: 1 when retrieval ran, 0 for recent
 *              context only. */
typedef struct {
  int32_t n_recent;
  int32_t n_before;
  int32_t n_after;
  int32_t retrieved;
} ss_evidence_params;

/* Long-term clusters retrieved for each stream (Eq. selected_cluster_evidence),
 * to unite with the detailed evidence.
 *   sets         host array of n_streams cluster sets (an entry may be NULL:
 *                that stream has no long-term memory);
 *   cluster_ids  device int64 [n_streams][k_clusters] cluster ids in any order,
 *                as ss_clusters_retrieve writes them (entries < 0, or of
 *                clusters not in use, are padding);
 *   k_clusters   1..64. */
typedef struct {
  const ss_clusters* const* sets;
  const int64_t* cluster_ids;
  int32_t k_clusters;
} ss_evidence_clusters;

/* Items ss_assemble_evidence can return per stream: n_recent, plus, when
 * retrieved, n_select*(1+n_before+n_after) + k_clusters (k_clusters = 0 without
 * clusters).  0 if the parameters are invalid or the count exceeds 4096. */
int32_t ss_evidence_max_units(const ss_evidence_params* params, int32_t n_select, int32_t k_clusters);

/* The evidence handed to full-depth answering for each of n_streams streams:
 * E_det(q) of Eq. selected_evidence united with E_cl(q) of Eq.
 * selected_cluster_evidence, deduplicated and in temporal order.  With T the
 * frames stored in idx[s] and D = [first_detail, T) its detailed window (all
 * of [0, T) unless frames left it through ss_clusters_absorb): the newest
 * min(n_recent, T) frames and, when retrieved, frames t-n_before .. t+n_after
 * of every selected frame t, each kept only if it lies in D (a frame that
 * left D exists only inside its cluster's representative); then, when
 * retrieved and clusters is given, every distinct retrieved cluster of the
 * stream, placed in the temporal order at its first member frame (clusters
 * cover disjoint runs of frames before D).
 *   frame_ids  device int64 [n_streams][n_select] as ss_retrieve writes them
 *              (entries < 0 are padding; ids >= T are skipped).  Not read, and
 *              may be NULL, when params->retrieved is 0.
 *   clusters   NULL for detailed evidence only; not read when not retrieved.
 *   units      device int64 [n_streams][max_units] out: frame ids (kind 0) or
 *              cluster ids (kind 1) in temporal order, -1 padded;
 *   kinds      device int32 [n_streams][max_units] out: 0 frame, 1 cluster,
 *              -1 padding; may be NULL when clusters is NULL;
 *   n_units    device int32 [n_streams] out.
 *   max_units  >= ss_evidence_max_units(params, n_select, k_clusters).
 * Enqueued on `stream` after the retrievals that wrote frame_ids and
 * cluster_ids; uses the frame counts and detailed windows of the indices at
 * the time of the call. */
ss_status ss_assemble_evidence(ss_index* const* idx, int32_t n_streams, const int64_t* frame_ids,
                               int32_t n_select, const ss_evidence_clusters* clusters,
                               const ss_evidence_params* params, void* stream, int64_t* units, int32_t* kinds,
                               int32_t* n_units, int32_t max_units);

/* Every score of one list over rows [row0, row0+n_rows) of one index, with the
 * same arithmetic as ss_retrieve (parity only).  queries: host array of L_s
 * device pointers as in ss_retrieve.  out: device fp32 [n_rows].  With
 * head_mode 1 `q_head` is ignored and the list is the layer's head mean.
 * ws: device workspace of ss_debug_scores_workspace_bytes() bytes. */
size_t ss_debug_scores_workspace_bytes(const ss_index* idx);
ss_status ss_debug_scores(const ss_index* idx, const void* const* queries, int32_t n_q,
                          int32_t layer, int32_t q_head, int32_t head_mode, int64_t row0,
                          int64_t n_rows, float* out, void* ws, size_t ws_bytes, void* stream);

/* Copy the stored state out (parity only; any pointer may be NULL), for the
 * frames the arena stores, first_stored .. n_frames-1 (ss_index_window):
 *   rows_dev     bf16 [L_s][H_kv][n_rows][d] device;
 *   counts_dev   int32 [L_s][H_kv][n_rows] device (k-means member counts, 1 for raw rows);
 *   desc_dev     fp32 [n_frames - first_stored][H_kv*d] device descriptors;
 *   frame_offsets_host  int64 [n_frames - first_stored + 1] host row offsets
 *                in the arena. */
ss_status ss_index_export(const ss_index* idx, void* rows_dev, int32_t* counts_dev,
                          float* desc_dev, int64_t* frame_offsets_host, void* stream);

/* The sample plan ss_retrieve uses for one list of n_rows candidate rows and
 * top_k (parity only; host work only).  The streaming cut-off of the list is
 * the r-th largest score among m evenly spread sampled rows: sample u < m is
 * row (u * step + step / 2) >> 32 with step = floor(n_rows * 2^32 / m), in
 * unsigned 64-bit arithmetic.  out (host int32 [4]): m, r, the list's
 * candidate capacity (a batch uses the capacity of its longest list), and
 * the expected candidate count the plan aims at (0 when n_rows is 0).  With
 * m = n_rows every row is sampled and r = min(top_k, n_rows). */
ss_status ss_debug_sample_plan(int64_t n_rows, int32_t top_k, int32_t* out);

/* Optional timing hook for the streaming scoring kernel: when both are
 * non-NULL hipEvent_t handles, later ss_retrieve calls on this thread record
 * `ev_start` just before that kernel and `ev_stop` just after it, on the
 * call's stream.  NULL, NULL turns it off. */
ss_status ss_set_profile_events(void* ev_start, void* ev_stop);

const char* ss_status_string(ss_status status);
const char* ss_last_error(void); /* thread-local text of the last failure */
int32_t ss_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SHALLOWSTREAM_H */
