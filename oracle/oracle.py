"""Float64 NumPy oracle of ShallowStream's query-time evidence retrieval.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU baseline, never by the library.  It shares no code with the
HIP path.

What is computed, in the paper's order (Sec. 4.1 "Query-Agnostic Shallow Index
Construction" and Sec. 4.2 "Query-Time Answering"):

* index: per shallow layer the keys of every stored unit (Eq. shallow_streaming_cache),
  with each unit's row range; a unit descriptor per frame (Eq. memory_key);
  optional per-frame k-means compression of the stored rows (an extension of the
  optional compression idea of Sec. 4.1, specified by the workload: k-means with
  farthest-point seeding, see ``kmeans``);
* candidates: every unit except the newest ``n_recent`` (Eq. context_partition);
* token scores (Sec. 4.2, "Optional Evidence Retrieval"), per (layer, query
  head), with the text-token queries reduced by their mean: either the scaled
  Q-K logit of the question against every candidate key, or the attention
  probability (the softmax of those logits over the candidate rows); per head
  or averaged over heads (``score_lists``);
* top-k per list (Eq. token_vote_candidates), ties to the lower row position;
* one vote per selected token for its unit, and the selected tokens' summed
  list values as the unit's "attention mass" tie-breaker;
* a vote-ranked pool of ``pool_mult * K`` units, then greedy max-min diversity in
  descriptor space (the DivTopK of Eq. selected_evidence).

Readings of points the paper leaves open are listed in the module functions'
docstrings.  Arithmetic is float64 on bfloat16-decoded inputs: products of two
bfloat16 values are exact in float64.
"""
from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------
# bfloat16 decoding (inputs are raw 16-bit patterns)
# ---------------------------------------------------------------------------


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float64 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    out = (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if not np.all(np.isfinite(out)):
        raise ValueError("NaN or Inf in bfloat16 input")
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest bfloat16 (ties to even), returned as bit patterns.

    The exact float64 value is rounded once: ``x = n * 2**(e-8)`` with the
    8-bit significand ``n`` rounded half-to-even (no detour through float32).
    """
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("NaN or Inf cannot be rounded to bfloat16")
    a = np.abs(x)
    _, e = np.frexp(a)                               # a = m * 2**e, m in [0.5, 1)
    e = np.maximum(e, -125)                          # below the normal range the quantum is fixed
    q = np.ldexp(1.0, e - 8)
    n = a / q                                        # exact: scaling by a power of two
    fl = np.floor(n)
    r = n - fl
    up = (r > 0.5) | ((r == 0.5) & (np.fmod(fl, 2.0) == 1.0))
    y = (fl + up) * q
    if np.any(y >= 2.0 ** 128):
        raise OverflowError("value overflows bfloat16")
    bits = (y.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return np.where(np.signbit(x), bits | np.uint16(0x8000), bits).astype(np.uint16)


# ---------------------------------------------------------------------------
# Unit descriptor (Eq. memory_key)
# ---------------------------------------------------------------------------


def descriptor(last_layer_keys: np.ndarray) -> np.ndarray:
    """Eq. memory_key: mean over the unit's raw visual tokens of the final shallow
    layer keys, all KV heads flattened head-major, then L2-normalised.

    ``last_layer_keys``: float64 ``[H_kv][T][d]``.  Returns ``[H_kv * d]``.
    A zero mean stays zero (the normalisation is undefined there).
    """
    Hk, T, d = last_layer_keys.shape
    mean = last_layer_keys.mean(axis=1)          # [H_kv][d]
    vec = mean.reshape(Hk * d)                   # vec(): head-major flatten
    n = np.sqrt(np.dot(vec, vec))
    return vec / n if n > 0 else vec


def unit_mean_keys(frame_layer_keys) -> np.ndarray:
    """The unit's pooled keys: per shallow layer and KV head, the mean of its raw
    visual tokens' keys (the unnormalised means behind Eq. memory_key, at every
    layer).  ``frame_layer_keys``: per layer ``uint16 [H_kv][T][d]``.  Returns
    float64 ``[L][H_kv][d]``."""
    return np.stack([decode_bf16(k).mean(axis=1) for k in frame_layer_keys])


# ---------------------------------------------------------------------------
# Per-frame k-means compression (compression at append time)
# ---------------------------------------------------------------------------


def kmeans(X: np.ndarray, n_centroids: int, n_iters: int):
    """k-means of one frame's tokens at one (layer, KV head).

    Readings (the paper's own compression clusters whole units over time; this
    per-frame token rule is the workload's):
      * squared Euclidean distance;
      * farthest-point initialisation: the first centre is the token farthest
        from the frame mean, each next one the not-yet-chosen token with the
        largest distance to its nearest chosen centre; ties to the lower index;
      * exactly ``n_iters`` rounds of (assign to nearest centre, ties to the
        lower centre index; move each centre to the mean of its members, an
        empty centre stays where it is);
      * ``min(n_centroids, T)`` centres in farthest-point order;
      * counts are the member counts of the last assignment.

    Returns ``(centres [c][d] float64, counts [c] int, diag)`` where ``diag``
    holds the smallest relative decision margins: ``init_margin`` over the
    farthest-point argmax decisions and ``assign_margin`` over every point's
    nearest-centre decision in every round.
    """
    X = np.asarray(X, dtype=np.float64)
    T, d = X.shape
    c = min(n_centroids, T)
    mu = X.mean(axis=0)
    d_mu = ((X - mu) ** 2).sum(axis=1)
    init_margin = _argmax_margin(d_mu, np.ones(T, dtype=bool))
    first = int(np.argmax(d_mu))                 # first index of the maximum
    chosen = [first]
    is_chosen = np.zeros(T, dtype=bool)
    is_chosen[first] = True
    mind = ((X - X[first]) ** 2).sum(axis=1)
    while len(chosen) < c:
        avail = ~is_chosen
        init_margin = min(init_margin, _argmax_margin(mind, avail))
        cand = np.where(avail, mind, -np.inf)
        nxt = int(np.argmax(cand))
        chosen.append(nxt)
        is_chosen[nxt] = True
        mind = np.minimum(mind, ((X - X[nxt]) ** 2).sum(axis=1))
    C = X[chosen].copy()
    assign_margin = np.inf
    assign = np.zeros(T, dtype=np.int64)
    sse = []
    for _ in range(n_iters):
        D = ((X[:, None, :] - C[None, :, :]) ** 2).sum(axis=2)   # [T][c]
        assign = np.argmin(D, axis=1)                              # ties -> lower centre
        if c > 1:
            part = np.sort(D, axis=1)
            best, second = part[:, 0], part[:, 1]
            with np.errstate(divide="ignore", invalid="ignore"):
                rel = np.where(second > 0, (second - best) / second, np.inf)
            assign_margin = min(assign_margin, float(rel.min()))
        sse.append(float(D[np.arange(T), assign].sum()))
        for j in range(c):
            members = assign == j
            if members.any():
                C[j] = X[members].mean(axis=0)
    counts = np.bincount(assign, minlength=c)[:c] if n_iters > 0 else np.zeros(c, dtype=np.int64)
    diag = {"init_margin": init_margin, "assign_margin": assign_margin, "sse": sse,
            "order": chosen}
    return C, counts, diag


def _argmax_margin(v: np.ndarray, avail: np.ndarray) -> float:
    vals = np.sort(v[avail])[::-1]
    if vals.size < 2 or vals[0] <= 0:
        return np.inf if vals.size < 2 else 0.0
    return float((vals[0] - vals[1]) / vals[0])


# ---------------------------------------------------------------------------
# The index (Eq. shallow_streaming_cache, Eq. memory_key, Eq. context_partition)
# ---------------------------------------------------------------------------


class Index:
    """Shallow-layer key index of one stream.

    Rows of layer ``l`` and KV head ``g`` are kept as bfloat16 bit patterns in
    append order; frame ``t`` owns rows ``[row_start[t], row_start[t] + row_count[t])``
    in every (layer, KV head).  Frame ids are append order, from 0.
    """

    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 n_recent: int = 0):
        if n_q_heads % n_kv_heads:
            raise ValueError("query heads must be a multiple of KV heads")
        self.L, self.Hq, self.Hk, self.d = n_layers, n_q_heads, n_kv_heads, head_dim
        self.G = n_q_heads // n_kv_heads
        self.n_recent = n_recent
        self.first_detail = 0        # units before it were folded into long-term clusters
        self._chunks = [[] for _ in range(n_layers)]    # per layer: list of [H_kv][r][d] uint16
        self._rows_cache = None
        self.row_start: list[int] = []
        self.row_count: list[int] = []
        self.desc: list[np.ndarray] = []
        self.pooled: list[np.ndarray] = []               # per frame [L][H_kv][d] mean raw key
        self.counts: list[np.ndarray] = []               # per frame [L][H_kv][rows] member counts
        self.kmeans_diag: list = []

    @property
    def n_frames(self) -> int:
        return len(self.row_start)

    @property
    def n_rows(self) -> int:
        return (self.row_start[-1] + self.row_count[-1]) if self.row_start else 0

    def append(self, layer_keys, n_frames: int, n_tokens: int, compress=None) -> int:
        """Append ``n_frames`` frames of ``n_tokens`` tokens.

        ``layer_keys``: per layer a ``uint16 [H_kv][n_frames * n_tokens][d]`` array.
        ``compress``: ``None`` or ``(n_centroids, n_iters)``.
        The descriptor always uses the raw keys of the last shallow layer.
        """
        if len(layer_keys) != self.L:
            raise ValueError("one key array per shallow layer expected")
        for a in layer_keys:
            if a.shape != (self.Hk, n_frames * n_tokens, self.d):
                raise ValueError(f"bad key array shape {a.shape}")
        first = self.n_frames
        T = n_tokens
        for f in range(n_frames):
            sl = slice(f * T, (f + 1) * T)
            last = decode_bf16(layer_keys[self.L - 1][:, sl, :])
            self.desc.append(descriptor(last))
            self.pooled.append(unit_mean_keys([layer_keys[l][:, sl, :] for l in range(self.L)]))
            if compress is None:
                rows = [layer_keys[l][:, sl, :] for l in range(self.L)]
                cnt = np.ones((self.L, self.Hk, T), dtype=np.int64)
                diag = None
            else:
                n_c, n_it = compress
                c_eff = min(n_c, T)
                rows, cnt, diag = [], np.zeros((self.L, self.Hk, c_eff), dtype=np.int64), []
                for l in range(self.L):
                    r = np.empty((self.Hk, c_eff, self.d), dtype=np.uint16)
                    x = decode_bf16(layer_keys[l][:, sl, :])
                    for g in range(self.Hk):
                        C, counts, dg = kmeans(x[g], n_c, n_it)
                        r[g] = round_bf16(C)
                        cnt[l, g] = counts
                        diag.append(dg)
                    rows.append(r)
            n_r = rows[0].shape[1]
            self.row_start.append(self.n_rows)
            self.row_count.append(n_r)
            for l in range(self.L):
                self._chunks[l].append(np.ascontiguousarray(rows[l]))
            self.counts.append(cnt)
            self.kmeans_diag.append(diag)
        self._rows_cache = None
        return first

    def append_stored(self, layer_rows, rows_per_frame, descriptors, pooled=None) -> int:
        """Append frames whose stored rows and descriptors were produced elsewhere
        (e.g. compressed rows exported from another implementation), so retrieval
        can be checked on identical stored data.

        ``layer_rows``: per layer ``uint16 [H_kv][sum(rows_per_frame)][d]``;
        ``descriptors``: ``[n_frames][H_kv * d]``; ``pooled``: optional
        ``[n_frames][L][H_kv][d]`` mean raw keys (``unit_mean_keys``).
        """
        first = self.n_frames
        start = 0
        for f, n_r in enumerate(rows_per_frame):
            self.desc.append(np.asarray(descriptors[f], dtype=np.float64))
            self.pooled.append(None if pooled is None else np.asarray(pooled[f], dtype=np.float64))
            self.row_start.append(self.n_rows)
            self.row_count.append(int(n_r))
            for l in range(self.L):
                self._chunks[l].append(np.ascontiguousarray(layer_rows[l][:, start:start + n_r, :]))
            self.counts.append(None)
            self.kmeans_diag.append(None)
            start += n_r
        self._rows_cache = None
        return first

    def rows(self, layer: int) -> np.ndarray:
        """All stored rows of a layer: ``uint16 [H_kv][N][d]``."""
        if self._rows_cache is None:
            self._rows_cache = [None] * self.L
        if self._rows_cache[layer] is None:
            ch = self._chunks[layer]
            self._rows_cache[layer] = (np.concatenate(ch, axis=1) if ch else
                                       np.zeros((self.Hk, 0, self.d), dtype=np.uint16))
        return self._rows_cache[layer]

    def candidate_frames(self) -> int:
        """Eq. context_partition: the newest ``n_recent`` units are never candidates."""
        return max(0, self.n_frames - self.n_recent)

    def candidate_rows(self) -> int:
        """End of the candidate rows (the rows before the recent window)."""
        f = self.candidate_frames()
        return self.row_start[f - 1] + self.row_count[f - 1] if f > 0 else 0

    def first_candidate_frame(self) -> int:
        """Units before ``first_detail`` left the detailed window: with long-history
        compression the token candidates are the detailed history S_T only
        (Eq. optional_context_compression; Sec. 4.2 takes candidates from S_T)."""
        return min(self.first_detail, self.candidate_frames())

    def first_candidate_row(self) -> int:
        f = self.first_candidate_frame()
        return self.row_start[f] if f < self.n_frames else self.n_rows

    def frame_of_row(self) -> np.ndarray:
        n = self.n_rows
        out = np.empty(n, dtype=np.int64)
        for t, (s, c) in enumerate(zip(self.row_start, self.row_count)):
            out[s:s + c] = t
        return out


# ---------------------------------------------------------------------------
# Query-time stages (Sec. 4.2, "Optional Evidence Retrieval")
# ---------------------------------------------------------------------------


def query_means(queries) -> list[np.ndarray]:
    """Per layer the mean over text tokens of each head's query: ``[H_q][d]`` float64."""
    return [decode_bf16(q).mean(axis=1) for q in queries]


def score_lists(index: Index, queries, head_mode: int = 0, score_mode: int = 0,
                chunk_rows: int = 1 << 16):
    """Token scores of every candidate row.

    Reading of multi-token questions: the paper scores with the final prompt
    token; with several text tokens the logit of a row is the mean over tokens
    of the scaled logit ``q_j . K_p / sqrt(d)``, which equals
    ``mean_j(q_j) . K_p / sqrt(d)`` and is the paper's logit when there is one
    token.  Keys and queries are taken as already rotated (RoPE upstream).
    Query head ``h`` reads KV head ``h // G``.

    ``score_mode == 0``: the value of a row in list (l, h) is that scaled logit.
    ``score_mode == 1``: the attention the question pays to the row (Sec. 4.2
    scores candidates by Q-K attention): the softmax of the list's logits over
    the candidate rows, ``exp(s_p - lse)`` with ``lse = log sum_p' exp(s_p')``
    over every candidate row ``p'`` of that (layer, query head).

    ``head_mode == 0``: one list per (layer, query head), ordered layer-major.
    ``head_mode == 1``: one list per layer, the values averaged over all query
    heads (Eq. token_vote_candidates averages over attention heads).  Under
    ``score_mode == 1`` each head is normalised by its own softmax before the
    average, so the two score modes rank rows differently in this head mode.

    Returns a list of float64 arrays over the candidate rows; position p is
    row ``index.first_candidate_row() + p``.
    """
    if head_mode not in (0, 1):
        raise ValueError("head_mode must be 0 or 1")
    if score_mode not in (0, 1):
        raise ValueError("score_mode must be 0 or 1")
    lo = index.first_candidate_row()
    N = index.candidate_rows() - lo
    scale = 1.0 / math.sqrt(index.d)
    qm = query_means(queries)
    lists = []
    for l in range(index.L):
        K = index.rows(l)
        per_head = np.empty((index.Hq, N))
        for g in range(index.Hk):
            Qg = qm[l][g * index.G:(g + 1) * index.G]          # [G][d]
            for r0 in range(0, N, chunk_rows):
                r1 = min(N, r0 + chunk_rows)
                Kc = decode_bf16(K[g, lo + r0:lo + r1, :])      # [r][d]
                per_head[g * index.G:(g + 1) * index.G, r0:r1] = (Kc @ Qg.T).T * scale
        if score_mode == 1 and N > 0:
            per_head = softmax_rows(per_head)
        if head_mode == 0:
            lists.extend(per_head[h] for h in range(index.Hq))
        else:
            lists.append(per_head.mean(axis=0))
    return lists


def softmax_rows(x: np.ndarray) -> np.ndarray:
    """Softmax of each row of ``x`` (shifted by the row maximum, which leaves the
    value unchanged and keeps ``exp`` finite)."""
    m = x.max(axis=1, keepdims=True)
    e = np.exp(x - m)
    return e / e.sum(axis=1, keepdims=True)


def score_scale(index: Index, queries, layer: int, q_head: int) -> np.ndarray:
    """Per candidate row the magnitude ``(1/sqrt d) * sum_e |qbar_e| |K_e|`` of its
    score's terms (the natural scale for score tolerances)."""
    lo, hi = index.first_candidate_row(), index.candidate_rows()
    qm = np.abs(query_means(queries)[layer][q_head])
    K = np.abs(decode_bf16(index.rows(layer)[q_head // index.G, lo:hi, :]))
    return (K @ qm) / math.sqrt(index.d)


def topk(scores: np.ndarray, k: int) -> np.ndarray:
    """Eq. token_vote_candidates: the ``min(k, N)`` rows of largest score; equal
    scores are ordered by the lower row position.  Returned in rank order."""
    order = np.argsort(-scores, kind="stable")     # stable: equal scores keep position order
    return order[:min(k, scores.size)]


def votes_and_mass(index: Index, topk_lists, score_lists_):
    """One vote per selected token for the unit that owns it (the vote count
    ``v_t``), and the unit's attention mass: the sum of its selected tokens'
    list values (scaled logits, or attention probabilities under
    ``score_mode == 1``), accumulated in (list, rank) order.

    Returns ``(votes [F] int64, mass [F] float64)`` over all frames.
    """
    F = index.n_frames
    f_of = index.frame_of_row()[index.first_candidate_row():index.candidate_rows()]
    votes = np.zeros(F, dtype=np.int64)
    mass = np.zeros(F, dtype=np.float64)
    for pos, s in zip(topk_lists, score_lists_):
        fr = f_of[pos]
        np.add.at(votes, fr, 1)
        np.add.at(mass, fr, s[pos])                 # unbuffered, in rank order
    return votes, mass


def vote_pool(votes: np.ndarray, mass: np.ndarray, size: int) -> np.ndarray:
    """Vote-ranked pool: units with at least one vote, ordered by (votes desc,
    mass desc, frame id asc), truncated to ``size``."""
    t = np.arange(votes.size)
    voted = votes >= 1
    idx = t[voted]
    order = np.lexsort((idx, -mass[voted], -votes[voted]))
    return idx[order][:size]


def maxmin_select(pool: np.ndarray, desc: np.ndarray, K: int):
    """Greedy max-min diversity over descriptors, seeded by the top of the vote
    ranking: each next unit maximises its smallest cosine distance ``1 - k_u.k_s``
    to the already selected units; ties go to the earlier pool rank.

    Returns ``(selected frame ids in selection order, margins)`` where
    ``margins[i]`` is the gap between the best and second-best candidate value
    at greedy step ``i`` (``inf`` when there was one candidate).
    """
    n = pool.size
    want = min(K, n)
    if want == 0:
        return np.zeros(0, dtype=np.int64), []
    D = desc[pool]                                   # [n][dim]
    sel = [0]
    taken = np.zeros(n, dtype=bool)
    taken[0] = True
    mind = 1.0 - D @ D[0]
    margins = []
    while len(sel) < want:
        cand = np.where(taken, -np.inf, mind)
        j = int(np.argmax(cand))                     # first maximum = earlier pool rank
        rest = np.sort(cand[~taken])[::-1]
        margins.append(float(rest[0] - rest[1]) if rest.size > 1 else np.inf)
        sel.append(j)
        taken[j] = True
        mind = np.minimum(mind, 1.0 - D @ D[j])
    return pool[np.array(sel)], margins


def retrieve(index: Index, queries, top_k: int, n_select: int, pool_mult: int = 4,
             head_mode: int = 0, debug: bool = False, score_mode: int = 0):
    """Evidence retrieval for one stream and one question.

    Returns ``(frame_ids, votes, mass, n_out)``: ``frame_ids`` in max-min
    selection order, padded with -1 to ``n_select``; ``votes``/``mass`` of the
    selected frames (0 in the padding).  With ``debug=True`` a dict of every
    intermediate is appended.
    """
    if top_k < 1 or n_select < 1 or pool_mult < 1:
        raise ValueError("top_k, n_select and pool_mult must be >= 1")
    S = score_lists(index, queries, head_mode, score_mode)
    T = [topk(s, top_k) for s in S]
    votes, mass = votes_and_mass(index, T, S)
    pool = vote_pool(votes, mass, pool_mult * n_select)
    desc = np.array(index.desc) if index.desc else np.zeros((0, index.Hk * index.d))
    sel, margins = maxmin_select(pool, desc, n_select)
    frame_ids = np.full(n_select, -1, dtype=np.int64)
    v_out = np.zeros(n_select, dtype=np.int64)
    m_out = np.zeros(n_select, dtype=np.float64)
    frame_ids[:sel.size] = sel
    v_out[:sel.size] = votes[sel]
    m_out[:sel.size] = mass[sel]
    out = (frame_ids, v_out, m_out, int(sel.size))
    if debug:
        return out + ({"scores": S, "topk": T, "votes": votes, "mass": mass, "pool": pool,
                       "maxmin_margins": margins},)
    return out


# ---------------------------------------------------------------------------
# Evidence assembly (Eq. selected_evidence, then deduplication and temporal
# ordering, Sec. 4.2)
# ---------------------------------------------------------------------------


def evidence_units(n_frames: int, selected, n_recent: int, n_before: int = 1, n_after: int = 0,
                   retrieved: bool = True, first_detail: int = 0) -> np.ndarray:
    """The detailed units handed to full-depth answering, ascending, without
    repeats (Eq. selected_evidence, then deduplication and temporal ordering).

    ``R_T`` is the newest ``n_recent`` units of the ``n_frames`` stored so far
    (Eq. context_partition).  When retrieval ran, each selected unit ``t`` is
    expanded to its temporal neighbours ``t - n_before .. t + n_after`` (the
    paper's setting is one preceding unit), and the evidence is ``R_T`` united
    with those; otherwise it is ``R_T`` alone.  Entries of ``selected`` below 0
    are padding and are ignored.

    Reading: every detailed unit lies in the detailed window ``[first_detail,
    n_frames)``: units that left it for long-term clusters (Eq.
    optional_context_compression) no longer exist on their own, only inside
    their cluster's representative, so neighbours and recent units below it
    are dropped (``first_detail`` is 0 without compression).
    """
    if n_frames < 0 or n_recent < 0 or n_before < 0 or n_after < 0 or first_detail < 0:
        raise ValueError("sizes must be >= 0")
    lo = min(first_detail, n_frames)
    units = set(range(max(lo, n_frames - n_recent), n_frames))
    if retrieved:
        for t in selected:
            t = int(t)
            if t < 0:
                continue
            if t >= n_frames:
                raise ValueError(f"selected unit {t} outside the {n_frames} stored units")
            for u in range(t - n_before, t + n_after + 1):
                if lo <= u < n_frames:
                    units.add(u)
    return np.array(sorted(units), dtype=np.int64)


def evidence_items(n_frames: int, selected, n_recent: int, n_before: int = 1, n_after: int = 0,
                   retrieved: bool = True, first_detail: int = 0, cluster_first=(),
                   selected_clusters=()):
    """``E_det(q)`` united with ``E_cl(q)`` after deduplication and temporal
    ordering (Eq. selected_evidence, Eq. selected_cluster_evidence and the
    sentence after it).

    ``cluster_first[j]`` is the first member unit of long-term cluster ``j``;
    ``selected_clusters`` the retrieved cluster ids (entries below 0, or not
    below ``len(cluster_first)``, are padding).  Reading: a cluster stands in
    the temporal order at its first member unit; the clusters cover disjoint
    runs of units before the detailed window, so no cluster and detailed unit
    share a position.  Without retrieval ``E_cl`` is empty.

    Returns ``(ids, kinds)``: int64 arrays in temporal order, kind 0 for a
    detailed unit (id = unit), kind 1 for a cluster (id = cluster).
    """
    det = evidence_units(n_frames, selected, n_recent, n_before, n_after, retrieved, first_detail)
    items = [(int(t), 0, int(t)) for t in det]
    if retrieved:
        seen = set()
        for j in selected_clusters:
            j = int(j)
            if j < 0 or j >= len(cluster_first) or j in seen:
                continue
            seen.add(j)
            items.append((int(cluster_first[j]), 1, j))
    items.sort()
    return (np.array([i for _, _, i in items], dtype=np.int64),
            np.array([k for _, k, _ in items], dtype=np.int64))


# ---------------------------------------------------------------------------
# Pooled shallow Q-K ranker (the baseline evidence ranker of the ablation
# comparing rankers in Sec. 5)
# ---------------------------------------------------------------------------


def pooled_scores(index: Index, queries) -> np.ndarray:
    """Score of every candidate unit under pooled shallow Q-K ranking.

    Reading: keys are pooled per unit before the Q-K product, so a unit's score
    is the scaled logit of the question's mean query against the unit's mean
    raw key (``unit_mean_keys``), averaged over every shallow layer and query
    head (query head ``h`` reads KV head ``h // G``):
    ``(1 / (L H_q)) sum_{l,h} qbar_{l,h} . Kbar_{l,g(h),t} / sqrt(d)``.  For raw
    units this is the mean of the unit's token scores over its tokens and over
    every (layer, head) list.  Candidates are the units before the recent window
    (Eq. context_partition) that are still in the detailed history; entry i
    belongs to unit ``index.first_candidate_frame() + i``.
    """
    f0, F = index.first_candidate_frame(), index.candidate_frames()
    qm = query_means(queries)
    s = np.zeros(F - f0)
    if F == f0:
        return s
    if any(p is None for p in index.pooled[f0:F]):
        raise ValueError("pooled keys missing for some units")
    Kp = np.stack(index.pooled[f0:F])                       # [F - f0][L][H_kv][d]
    for l in range(index.L):
        for h in range(index.Hq):
            s += Kp[:, l, h // index.G, :] @ qm[l][h]
    return s / (index.L * index.Hq * math.sqrt(index.d))


def pooled_retrieve(index: Index, queries, n_select: int):
    """The ``n_select`` best units by pooled score, ties to the earlier unit; no
    diversity selection or temporal expansion.  Returns ``(frame_ids, scores,
    n_out)`` padded with -1 and 0."""
    if n_select < 1:
        raise ValueError("n_select must be >= 1")
    s = pooled_scores(index, queries)
    t = np.arange(s.size)
    order = np.lexsort((t, -s))[:n_select]
    ids = np.full(n_select, -1, dtype=np.int64)
    sc = np.zeros(n_select)
    ids[:order.size] = order + index.first_candidate_frame()
    sc[:order.size] = s[order]
    return ids, sc, int(order.size)


# ---------------------------------------------------------------------------
# Long-history compression (Sec. 4.1, "Optional Long-History Compression") and
# cluster retrieval (Eq. selected_cluster_evidence)
# ---------------------------------------------------------------------------


class LongClusters:
    """Long-term clusters of the units that left the detailed window.

    Units leave in temporal order.  Eq. optional_long_memory_clustering: a
    leaving unit ``t`` joins the latest cluster ``C_j`` when its descriptor
    ``k_t`` (Eq. memory_key) satisfies ``k_t . c_j >= tau``, and then
    ``c_j <- Norm((n_j c_j + k_t) / (n_j + 1))``; otherwise it starts a new
    cluster with ``c = k_t``.  Eq. optional_long_memory_representative: the
    cluster's representative keys are the running average
    ``(n_j Kbar_j + K_t) / (n_j + 1)`` of the members' stored rows, position by
    position, at every shallow layer.

    Readings: the threshold and budget are parameters (the paper gives no
    values); ``Norm`` of a zero vector stays zero; when ``max_clusters`` are in
    use a unit that would open a new cluster joins the latest one instead and
    ``overflow`` is set.
    """

    def __init__(self, tau: float, max_clusters: int):
        if max_clusters < 1:
            raise ValueError("max_clusters must be >= 1")
        self.tau, self.max_clusters = float(tau), int(max_clusters)
        self.centroids: list[np.ndarray] = []
        self.sizes: list[int] = []
        self.first: list[int] = []
        self.last: list[int] = []
        self.rep: list[np.ndarray] = []     # per cluster [L][H_kv][rows][d] float64
        self.overflow = False
        self.margins: list[float] = []      # |k_t . c - tau| of every join decision

    def absorb(self, index: Index, frame_hi: int) -> None:
        """Units ``index.first_detail .. frame_hi - 1`` leave the detailed window."""
        f0 = index.first_detail
        if not f0 <= frame_hi <= index.candidate_frames():
            raise ValueError("units leave in order and never from the recent window")
        for t in range(f0, frame_hi):
            k = index.desc[t]
            r0, n_r = index.row_start[t], index.row_count[t]
            K_t = np.stack([decode_bf16(index.rows(l)[:, r0:r0 + n_r, :]) for l in range(index.L)])
            if self.rep and K_t.shape != self.rep[0].shape:
                raise ValueError("every clustered unit must store the same number of rows")
            joins = False
            if self.centroids:
                dot = float(k @ self.centroids[-1])
                joins = dot >= self.tau
                self.margins.append(abs(dot - self.tau))
            if not joins and self.centroids and len(self.centroids) == self.max_clusters:
                joins = True
                self.overflow = True
            if joins:
                n = self.sizes[-1]
                c = (n * self.centroids[-1] + k) / (n + 1)
                norm = math.sqrt(float(c @ c))
                self.centroids[-1] = c / norm if norm > 0 else c
                self.rep[-1] = (n * self.rep[-1] + K_t) / (n + 1)
                self.sizes[-1] = n + 1
                self.last[-1] = t
            else:
                self.centroids.append(np.array(k, dtype=np.float64))
                self.rep.append(K_t)
                self.sizes.append(1)
                self.first.append(t)
                self.last.append(t)
        index.first_detail = frame_hi


def frame_bytes(n_rows: int, n_layers: int, n_kv_heads: int, head_dim: int) -> int:
    """Index bytes one stored unit takes: its keys (bfloat16) and member counts
    (int32) at every shallow layer and KV head, its descriptor (Eq. memory_key)
    and pooled keys (float32), and its row offset (int32)."""
    return (n_rows * n_layers * n_kv_heads * (2 * head_dim + 4)
            + (1 + n_layers) * n_kv_heads * head_dim * 4 + 4)


def budget_split(row_counts, first_detail: int, n_recent: int, n_layers: int, n_kv_heads: int,
                 head_dim: int, budget: int) -> int:
    """Eq. optional_context_compression: once the memory of the detailed history
    exceeds the budget B, the oldest detailed units leave for long-term
    clusters while the recent context stays detailed.  Reading: Mem is the
    index bytes (``frame_bytes``) of the units in the detailed window
    ``[first_detail, T)``; the result is the smallest ``h`` in
    ``[first_detail, max(first_detail, T - n_recent)]`` whose units ``[h, T)``
    fit in ``budget``, or the end of that range when none does."""
    T = len(row_counts)
    hi = max(first_detail, T - n_recent)
    for h in range(first_detail, hi + 1):
        mem = sum(frame_bytes(int(row_counts[f]), n_layers, n_kv_heads, head_dim) for f in range(h, T))
        if mem <= budget:
            return h
    return hi


def cluster_scores(index: Index, clusters: LongClusters, queries) -> np.ndarray:
    """Eq. selected_cluster_evidence scores every centroid against the final
    shallow query state.  Reading: the centroid lives in the descriptor space of
    Eq. memory_key (KV heads flattened head-major), so query head ``h`` of the
    last shallow layer meets the centroid's block of KV head ``h // G``; the
    score is the scaled logit averaged over query heads, with the question's
    tokens reduced by their mean as for token scores."""
    q = query_means(queries)[index.L - 1]                   # [H_q][d]
    C = np.array(clusters.centroids).reshape(-1, index.Hk, index.d)
    s = np.zeros(C.shape[0])
    for h in range(index.Hq):
        s += C[:, h // index.G, :] @ q[h]
    return s / (index.Hq * math.sqrt(index.d))


def cluster_retrieve(index: Index, clusters: LongClusters, queries, k_clusters: int):
    """TopK_{K_l} of the clusters by score, ties to the older cluster.
    Returns ``(cluster ids, scores, first frames, last frames, n_out)``, padded
    with -1 / 0."""
    if k_clusters < 1:
        raise ValueError("k_clusters must be >= 1")
    s = cluster_scores(index, clusters, queries) if clusters.centroids else np.zeros(0)
    order = np.lexsort((np.arange(s.size), -s))[:k_clusters]
    ids = np.full(k_clusters, -1, dtype=np.int64)
    sc = np.zeros(k_clusters)
    fst = np.full(k_clusters, -1, dtype=np.int64)
    lst = np.full(k_clusters, -1, dtype=np.int64)
    ids[:order.size] = order
    sc[:order.size] = s[order]
    fst[:order.size] = np.array(clusters.first)[order] if order.size else []
    lst[:order.size] = np.array(clusters.last)[order] if order.size else []
    return ids, sc, fst, lst, int(order.size)
