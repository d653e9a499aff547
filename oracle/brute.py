"""Pure-Python brute force of the same retrieval, for tiny inputs only.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Written independently of
``oracle.oracle``: plain loops, ``math.fsum`` for every sum, Python's ``sorted``
with explicit tuple keys, and token scores taken as the mean of the per-token
scaled logits (Sec. 4.2, "Optional Evidence Retrieval"), not a pre-averaged
query; attention probabilities from explicit exponentials of each list.  It
exists to cross-check the vectorised oracle.
"""
from __future__ import annotations

import math
import struct


def bf16_value(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def _vec(bits_row) -> list:
    return [bf16_value(b) for b in bits_row]


def _sqdist(a, b) -> float:
    return math.fsum((x - y) * (x - y) for x, y in zip(a, b))


def descriptor(frame_last_layer) -> list:
    """``frame_last_layer[g][t][e]`` floats -> unit descriptor (Eq. memory_key)."""
    Hk = len(frame_last_layer)
    T = len(frame_last_layer[0])
    d = len(frame_last_layer[0][0])
    flat = []
    for g in range(Hk):
        for e in range(d):
            flat.append(math.fsum(frame_last_layer[g][t][e] for t in range(T)) / T)
    norm = math.sqrt(math.fsum(x * x for x in flat))
    return [x / norm for x in flat] if norm > 0 else flat


def kmeans(X, n_centroids: int, n_iters: int):
    """Same rule as the oracle's: farthest-point seeding from the frame mean, then
    ``n_iters`` Lloyd rounds; ties to the lower index everywhere."""
    T = len(X)
    d = len(X[0])
    c = min(n_centroids, T)
    mu = [math.fsum(X[t][e] for t in range(T)) / T for e in range(d)]
    best_i, best_v = 0, -1.0
    for i in range(T):
        v = _sqdist(X[i], mu)
        if v > best_v:
            best_i, best_v = i, v
    chosen = [best_i]
    while len(chosen) < c:
        best_i, best_v = -1, -1.0
        for i in range(T):
            if i in chosen:
                continue
            v = min(_sqdist(X[i], X[j]) for j in chosen)
            if v > best_v:
                best_i, best_v = i, v
        chosen.append(best_i)
    C = [list(X[i]) for i in chosen]
    assign = [0] * T
    for _ in range(n_iters):
        for i in range(T):
            dists = [_sqdist(X[i], C[j]) for j in range(c)]
            assign[i] = min(range(c), key=lambda j: (dists[j], j))
        for j in range(c):
            mem = [X[i] for i in range(T) if assign[i] == j]
            if mem:
                C[j] = [math.fsum(m[e] for m in mem) / len(mem) for e in range(d)]
    counts = [sum(1 for i in range(T) if assign[i] == j) for j in range(c)] if n_iters else [0] * c
    return C, counts, chosen


def retrieve(frames, queries, n_kv_heads: int, top_k: int, n_select: int, pool_mult: int = 4,
             n_recent: int = 0, head_mode: int = 0, score_mode: int = 0):
    """Brute-force retrieval over raw (uncompressed) frames.

    ``frames[t][l][g][p]`` : list of bfloat16 bit rows (length d) of frame ``t``;
    ``queries[l][h][j]``   : bfloat16 bit rows of query token ``j`` of head ``h``.
    ``score_mode`` 1 turns each (layer, head)'s logits into attention
    probabilities over the candidate rows (``exp(s - lse)``, ``lse`` from the
    largest logit plus the log of an ``fsum`` of exponentials); ``head_mode`` 1
    averages the per-head values of a row over the layer's heads (one list per
    layer).  Returns ``(frame_ids, votes, mass, debug)`` with the padding of the
    oracle.
    """
    F = len(frames)
    L = len(queries)
    Hq = len(queries[0])
    G = Hq // n_kv_heads
    d = len(queries[0][0][0])
    F_c = max(0, F - n_recent)
    owner = []                     # frame of each candidate row, in append order
    for t in range(F_c):
        owner.extend([t] * len(frames[t][0][0]))
    lists = []
    for l in range(L):
        per_head = []
        for h in range(Hq):
            g = h // G
            qs = [_vec(qj) for qj in queries[l][h]]
            vals = []
            for t in range(F_c):
                for krow in frames[t][l][g]:
                    k = _vec(krow)
                    logits = [math.fsum(a * b for a, b in zip(q, k)) / math.sqrt(d) for q in qs]
                    vals.append(math.fsum(logits) / len(logits))
            if score_mode == 1 and vals:
                top = max(vals)
                lse = top + math.log(math.fsum(math.exp(v - top) for v in vals))
                vals = [math.exp(v - lse) for v in vals]
            per_head.append(vals)
        if head_mode == 0:
            row_lists = per_head
        else:
            n = len(owner)
            row_lists = [[math.fsum(per_head[h][p] for h in range(Hq)) / Hq for p in range(n)]]
        for vals in row_lists:
            scored = [(v, owner[p], p) for p, v in enumerate(vals)]
            ranked = sorted(scored, key=lambda x: (-x[0], x[2]))
            lists.append(ranked[:min(top_k, len(ranked))])
    votes = [0] * F
    contrib = [[] for _ in range(F)]
    for lst in lists:
        for s, t, _ in lst:
            votes[t] += 1
            contrib[t].append(s)
    mass = [math.fsum(c) for c in contrib]
    voted = [t for t in range(F) if votes[t] >= 1]
    pool = sorted(voted, key=lambda t: (-votes[t], -mass[t], t))[:pool_mult * n_select]
    descs = []
    for t in range(F):
        last = [[_vec(r) for r in frames[t][L - 1][g]] for g in range(n_kv_heads)]
        descs.append(descriptor(last))
    sel = []
    if pool:
        sel = [pool[0]]
        while len(sel) < min(n_select, len(pool)):
            best, best_v = None, -math.inf
            for u in pool:                       # pool order: first maximum wins
                if u in sel:
                    continue
                v = min(1.0 - math.fsum(a * b for a, b in zip(descs[u], descs[s])) for s in sel)
                if v > best_v:
                    best, best_v = u, v
            sel.append(best)
    ids = sel + [-1] * (n_select - len(sel))
    vo = [votes[t] for t in sel] + [0] * (n_select - len(sel))
    ma = [mass[t] for t in sel] + [0.0] * (n_select - len(sel))
    return ids, vo, ma, {"lists": lists, "votes": votes, "mass": mass, "pool": pool,
                         "desc": descs}


def pooled_scores(frames, queries, n_kv_heads: int, n_recent: int = 0) -> list:
    """Pooled shallow Q-K score of every candidate unit, written out as the mean,
    over layers, query heads, query tokens and the unit's tokens, of the scaled
    per-token logit (``frames`` and ``queries`` as in ``retrieve``)."""
    F = len(frames)
    L = len(queries)
    Hq = len(queries[0])
    G = Hq // n_kv_heads
    d = len(queries[0][0][0])
    out = []
    for t in range(max(0, F - n_recent)):
        terms = []
        for l in range(L):
            for h in range(Hq):
                g = h // G
                toks = frames[t][l][g]
                qs = queries[l][h]
                w = 1.0 / (L * Hq * len(qs) * len(toks))
                for qj in qs:
                    q = _vec(qj)
                    for krow in toks:
                        k = _vec(krow)
                        terms.append(w * math.fsum(a * b for a, b in zip(q, k)) / math.sqrt(d))
        out.append(math.fsum(terms))
    return out
